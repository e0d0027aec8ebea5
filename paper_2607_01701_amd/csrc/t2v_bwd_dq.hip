// Backward dQ kernel: a workgroup owns a query tile of one (clip, head) and loops over
// the clip's keys; every output element is written by one lane (no atomics).
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

constexpr int kDqQB = 1;  // 32-query blocks per wave
constexpr int kDqBN = 64; // keys per LDS stage (a multiple of 32)
// Wide tiles: eight waves (256 queries) share each staged K/V tile; narrow tiles: four
// waves (128 queries), two workgroups per CU, for packs with short key segments.
constexpr int kDqThreadsWide = 512;
constexpr int kDqThreadsNarrow = 256;

// ------------------------------------------------------------------------ backward: dQ

// One 32-key step for this wave's QB query blocks. RAGGED: only the first nvalid keys of
// the step are inside the clip.
template <int D, int QB, bool RAGGED>
T2V_DEV void dq_step(uint32_t kbase, uint32_t vbase, uint32_t kr0, uint32_t kr1, int kb, int nvalid, float c,
                     const bf16x8 (&qop)[QB][D / 16],
                     const bf16x8 (&gop)[QB][D / 16], const float (&nl2)[QB], const float (&ndl)[QB],
                     f32x16 (&dqa)[QB][D / 32], int lane) {
  // Let the scheduler interleave this step's LDS reads with its MFMAs (measured: +2 to +4%).
  __builtin_amdgcn_iglp_opt(0);
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  // S^T and dP^T (32 keys x 32 queries): lane = query, register r = key kb + 8 (r/4) + 4 G + r % 4.
  f32x16 s[QB], dp[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    s[qb] = zero16();
    dp[qb] = zero16();
  }
  {
    bf16x8 ka[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) ka[kk] = read_opnd<D>(kbase, kb, kk);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) s[qb] = mfma(ka[kk], qop[qb][kk], s[qb]);
  }
  {
    bf16x8 va[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) va[kk] = read_opnd<D>(vbase, kb, kk);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) dp[qb] = mfma(va[kk], gop[qb][kk], dp[qb]);
  }
  bf16x8 kt[2][DB];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) kt[hf][db] = read_rows_opnd<D>(kr0, kr1, kb + hf * 16, db);
  bf16x8 sb[QB][2];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float p = __builtin_amdgcn_exp2f(fmaf(s[qb][r], c, nl2[qb]));
      if constexpr (RAGGED) {  // keys past the clip must not contribute
        const int key = (r >> 2) * 8 + G * 4 + (r & 3);
        p = key < nvalid ? p : 0.0f;
      }
      s[qb][r] = p * (dp[qb][r] + ndl[qb]);
    }
    sb[qb][0] = to_bf16x8(s[qb], 0);
    sb[qb][1] = to_bf16x8(s[qb], 8);
  }
  // dQ^T += K^T dS^T over the 16 keys of half hf.
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) dqa[qb][db] = mfma(kt[hf][db], sb[qb][hf], dqa[qb][db]);
}

template <int D, int QB, int NT, bool PERSIST>
__global__ __launch_bounds__(NT, 512 / NT) void attn_bwd_dq_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ ndelta,
    const Item* __restrict__ items, int H, int64_t T, float c, float scale, bf16* __restrict__ dq,
    unsigned long long* __restrict__ trace, int n_items) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  constexpr int BN = kDqBN;  // keys per LDS stage
  __shared__ __attribute__((aligned(1024))) bf16 sK[2][BN * D];
  __shared__ __attribute__((aligned(1024))) bf16 sV[2][BN * D];

  // One work item per workgroup, or (persistent grid) items w, w + grid, w + 2 grid, ...: the
  // grid is a multiple of the 8 XCDs, so every item still runs on XCD (item mod 8).
  for (int w = blockIdx.x, first = 1; PERSIST ? w < n_items : first != 0; w += gridDim.x, first = 0) {
    const unsigned long long trace_t0 = trace != nullptr ? trace_clock() : 0ull;
    const Item it = items[w];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int G = lane >> 5;
    const int l32 = lane & 31;
    const int Lq = it.len;   // queries of the sequence (this tile's rows)
    const int L = it.llen;   // keys of the sequence (the loop)
    const int64_t rs = static_cast<int64_t>(H) * D;
    const int64_t base = static_cast<int64_t>(it.row0) * rs + static_cast<int64_t>(it.head) * D;
    const int64_t kvbase = static_cast<int64_t>(it.lrow0) * rs + static_cast<int64_t>(it.head) * D;
    const int64_t lbase = static_cast<int64_t>(it.head) * T + it.row0;
    const bf16* kh = k + kvbase;
    const bf16* vh = v + kvbase;
    const int q_wave0 = it.tile0 + wave * QB * 32;
    const bool wave_active = q_wave0 < Lq;

    const TileDma<D, BN, NT> dma(tid, rs);
    dma.copy(sK[0], kh, rs, 0, L);
    dma.copy(sV[0], vh, rs, 0, L);

    bf16x8 qop[QB][KK], gop[QB][KK];
    float nl2[QB], ndl[QB];  // -lse * log2(e) and -Delta of this lane's query
  #pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qi = q_wave0 + qb * 32 + l32;
      const bool ok = qi < Lq;
  #pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        qop[qb][kk] = load8(q + base + qi * rs + kk * 16 + G * 8, ok);
        gop[qb][kk] = load8(dout + base + qi * rs + kk * 16 + G * 8, ok);
      }
      nl2[qb] = ok ? -lse2[lbase + qi] : 0.0f;
      ndl[qb] = ok ? ndelta[lbase + qi] : 0.0f;
    }
    f32x16 dqa[QB][DB];
  #pragma unroll
    for (int qb = 0; qb < QB; ++qb)
  #pragma unroll
      for (int db = 0; db < DB; ++db) dqa[qb][db] = zero16();

    const int ntiles = (L + BN - 1) / BN;
    const int nfull = L / BN;
    const uint32_t oo = opnd_lane_off<D>(lane);
    const uint32_t ro0 = rows_lane_off<D>(lane, 0), ro1 = rows_lane_off<D>(lane, 1);
    wait_vmcnt0();
    __syncthreads();
    for (int tt = 0; tt < nfull; ++tt) {
      const int b = tt & 1;
      if (tt + 1 < ntiles) {
        dma.copy(sK[b ^ 1], kh, rs, (tt + 1) * BN, L);
        dma.copy(sV[b ^ 1], vh, rs, (tt + 1) * BN, L);
      }
      if (wave_active) {
        const uint32_t tk = lds_addr(sK[b]);
        const uint32_t kb0 = tk + oo, vb0 = lds_addr(sV[b]) + oo, k0 = tk + ro0, k1 = tk + ro1;
  #pragma unroll
        for (int kb = 0; kb < BN; kb += 32)
          dq_step<D, QB, false>(kb0, vb0, k0, k1, kb, 32, c, qop, gop, nl2, ndl, dqa, lane);
      }
      wait_vmcnt0();
      __syncthreads();
    }
    if (nfull < ntiles && wave_active) {
      const int b = nfull & 1;
      const int rem = L - nfull * BN;
      const uint32_t tk = lds_addr(sK[b]);
      const uint32_t kb0 = tk + oo, vb0 = lds_addr(sV[b]) + oo, k0 = tk + ro0, k1 = tk + ro1;
      // Every step of the last tile takes the masked form (a full step masks nothing): one
      // inlined copy instead of two keeps the tail within the register budget (the two-copy
      // tail spilled 34 VGPRs at D = 128; measured on short key segments: dQ -12%).
  #pragma unroll
      for (int kb = 0; kb < BN; kb += 32)
        if (rem > kb) dq_step<D, QB, true>(kb0, vb0, k0, k1, kb, min(rem - kb, 32), c, qop, gop, nl2, ndl, dqa, lane);
    }

    if (wave_active) {
  #pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int qi = q_wave0 + qb * 32 + l32;
        if (qi < Lq) {
          bf16* row = dq + base + qi * rs;
  #pragma unroll
          for (int db = 0; db < DB; ++db) {
  #pragma unroll
            for (int i = 0; i < 4; ++i) {
              bf16x4 w;
  #pragma unroll
              for (int e = 0; e < 4; ++e) w[e] = static_cast<bf16>(dqa[qb][db][i * 4 + e] * scale);
              *reinterpret_cast<bf16x4*>(row + db * 32 + i * 8 + G * 4) = w;
            }
          }
        }
      }
    }
    if (trace != nullptr) trace_end(trace, trace_t0, 3, w);
    if constexpr (PERSIST) {
      if (w + static_cast<int>(gridDim.x) < n_items) __syncthreads();  // LDS reads done before the next item's DMA
    }
  }
}

}  // namespace

int dq_tile_rows(int, bool narrow) { return ((narrow ? kDqThreadsNarrow : kDqThreadsWide) / 64) * 32 * kDqQB; }

namespace {
template <int D, int NT>
void launch_dq_as(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream) {
  const float c = a.scale * kLog2e;
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  const auto* g = static_cast<const bf16*>(a.dout);
  auto* dq = static_cast<bf16*>(a.dq);
  const float* lse2 = a.delta + a.total_tokens * a.heads;
  // Always one workgroup per item: the persistent form of this kernel needs more than the 256
  // registers per lane its two waves per SIMD allow, and spills (rejected by the build).
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, kDqQB, NT, false>), dim3(n_items), dim3(NT), 0, stream, q, k, v, g, lse2,
                     a.delta, items, a.heads, a.total_tokens, c, a.scale, dq, a.trace, n_items);
}
}  // namespace

hipError_t launch_bwd_dq(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream) {
  const bool narrow = a.q_rows == dq_tile_rows(a.head_dim, true);
  if (!narrow && a.q_rows != dq_tile_rows(a.head_dim, false)) return hipErrorInvalidValue;
  if (a.head_dim == 128) {
    if (narrow)
      launch_dq_as<128, kDqThreadsNarrow>(a, items, n_items, stream);
    else
      launch_dq_as<128, kDqThreadsWide>(a, items, n_items, stream);
  } else {
    if (narrow)
      launch_dq_as<64, kDqThreadsNarrow>(a, items, n_items, stream);
    else
      launch_dq_as<64, kDqThreadsWide>(a, items, n_items, stream);
  }
  return hipGetLastError();
}
#if T2V_CHECKED
hipError_t dq_check_take(unsigned int* rec, unsigned int canary) { return kern::check_take_here(rec, canary); }
#endif
}  // namespace t2v
