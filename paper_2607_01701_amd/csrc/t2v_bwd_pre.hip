// Backward preprocess: -Delta = -rowsum(dO * O) and lse * log2(e) (HBM-bound).
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

// ------------------------------------------------------------------- backward: Delta

// ndelta[h, t] = -sum_d dO[t, h, d] O[t, h, d]  and  lse2[h, t] = lse[h, t] * log2(e). Delta is
// stored negated because the dK/dV kernel starts its dP accumulator from it (dP - Delta
// then costs no subtraction) and the dQ kernel adds it.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_bwd_pre_kernel(const bf16* __restrict__ out,
                                                                 const bf16* __restrict__ dout,
                                                                 const float* __restrict__ lse, int64_t rows,
                                                                 int H, int64_t T, float* __restrict__ ndelta,
                                                                 float* __restrict__ lse2) {
  constexpr int LPR = D / 8;            // lanes per (token, head) row
  constexpr int RPB = kThreads / LPR;   // rows per workgroup step
  const int sub = threadIdx.x % LPR;
  for (int64_t row = static_cast<int64_t>(blockIdx.x) * RPB + threadIdx.x / LPR; row < rows;
       row += static_cast<int64_t>(gridDim.x) * RPB) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(out + row * D + sub * 8);
    const bf16x8 g = *reinterpret_cast<const bf16x8*>(dout + row * D + sub * 8);
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc = fmaf(static_cast<float>(a[t]), static_cast<float>(g[t]), acc);
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, LPR);
    if (sub == 0) {
      const int64_t t = row / H;
      const int64_t h = row - t * H;
      ndelta[h * T + t] = -acc;
      lse2[h * T + t] = lse[h * T + t] * kLog2e;
    }
  }
}


}  // namespace

hipError_t launch_bwd_pre(const AttnArgs& a, hipStream_t stream) {
  const int64_t rows = a.total_tokens * a.heads;
  const int lpr = a.head_dim / 8;
  const int64_t rpb = kThreads / lpr;
  const int64_t want = (rows + rpb - 1) / rpb;
  const dim3 grid(static_cast<unsigned>(want < 8192 ? want : 8192)), block(kThreads);
  const auto* o = static_cast<const bf16*>(a.out);
  const auto* g = static_cast<const bf16*>(a.dout);
  float* lse2 = a.delta + rows;
  if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_bwd_pre_kernel<128>), grid, block, 0, stream, o, g, a.lse, rows, a.heads,
                       a.total_tokens, a.delta, lse2);
  else
    hipLaunchKernelGGL((attn_bwd_pre_kernel<64>), grid, block, 0, stream, o, g, a.lse, rows, a.heads,
                       a.total_tokens, a.delta, lse2);
  return hipGetLastError();
}
}  // namespace t2v
