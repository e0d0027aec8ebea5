// Backward preprocess: -Delta = -rowsum(dO * O) and lse * log2(e) (HBM-bound).
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

// ------------------------------------------------------------------- backward: Delta

// ndelta[h, t] = -sum_d dO[t, h, d] O[t, h, d]  and  lse2[h, t] = lse[h, t] * log2(e). Delta is
// stored negated because the dK/dV kernel starts its dP accumulator from it (dP - Delta
// then costs no subtraction) and the dQ kernel adds it.
//
// A workgroup owns one head and kPreTokens consecutive tokens: D / 8 lanes read one
// (token, head) row of O and dO (16 bytes each per lane, the row contiguous), the row sums
// go through LDS, and the [H, T] outputs leave as contiguous runs of kPreTokens floats (the
// lse reads likewise), rather than as 4-byte accesses T floats apart.
constexpr int kPreTokens = 64;

template <int D>
__global__ __launch_bounds__(kThreads) void attn_bwd_pre_kernel(const bf16* __restrict__ out,
                                                                 const bf16* __restrict__ dout,
                                                                 const float* __restrict__ lse, int H,
                                                                 int64_t T, float* __restrict__ ndelta,
                                                                 float* __restrict__ lse2) {
  constexpr int LPR = D / 8;                 // lanes per (token, head) row
  constexpr int RPI = kThreads / LPR;        // rows per pass of the workgroup
  constexpr int NPASS = kPreTokens / RPI;    // passes per tile
  static_assert(kPreTokens % RPI == 0 && kPreTokens <= kThreads, "whole passes; one store lane per token");
  __shared__ float sres[kPreTokens];
  const int64_t ntb = (T + kPreTokens - 1) / kPreTokens;  // token blocks per head
  const int64_t h = static_cast<int64_t>(blockIdx.x) / ntb;
  const int64_t t0 = (static_cast<int64_t>(blockIdx.x) - h * ntb) * kPreTokens;
  const int sub = threadIdx.x % LPR;
  const int r = threadIdx.x / LPR;
  const int64_t rs = static_cast<int64_t>(H) * D;
  bf16x8 a[NPASS], g[NPASS];
#pragma unroll
  for (int i = 0; i < NPASS; ++i) {
    const int64_t t = t0 + i * RPI + r;
    const bool ok = t < T;
    const int64_t off = (ok ? t : 0) * rs + h * D + sub * 8;
    a[i] = load8(out + off, ok);
    g[i] = load8(dout + off, ok);
  }
#pragma unroll
  for (int i = 0; i < NPASS; ++i) {
    float acc = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(static_cast<float>(a[i][e]), static_cast<float>(g[i][e]), acc);
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, LPR);
    if (sub == 0) sres[i * RPI + r] = acc;
  }
  __syncthreads();
  const int64_t t = t0 + threadIdx.x;
  if (threadIdx.x < kPreTokens && t < T) {
    ndelta[h * T + t] = -sres[threadIdx.x];
    lse2[h * T + t] = lse[h * T + t] * kLog2e;
  }
}


}  // namespace

hipError_t launch_bwd_pre(const AttnArgs& a, hipStream_t stream) {
  const int64_t rows = a.total_tokens * a.heads;
  const int64_t ntb = (a.total_tokens + kPreTokens - 1) / kPreTokens;
  const dim3 grid(static_cast<unsigned>(ntb * a.heads)), block(kThreads);
  const auto* o = static_cast<const bf16*>(a.out);
  const auto* g = static_cast<const bf16*>(a.dout);
  float* lse2 = a.delta + rows;
  if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_bwd_pre_kernel<128>), grid, block, 0, stream, o, g, a.lse, a.heads, a.total_tokens,
                       a.delta, lse2);
  else
    hipLaunchKernelGGL((attn_bwd_pre_kernel<64>), grid, block, 0, stream, o, g, a.lse, a.heads, a.total_tokens,
                       a.delta, lse2);
  return hipGetLastError();
}
}  // namespace t2v
