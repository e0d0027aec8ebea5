// Backward dK/dV kernel: a workgroup owns 128 keys of one (clip, head) and loops over
// the clip's queries (see t2v_fwd.hip for the shared design notes).
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

constexpr int kDkdvBM = 64;  // queries per LDS stage (a multiple of 32)

// Asynchronous copy of 64 consecutive floats (rows row0 .. row0 + 63, clamped to L - 1)
// into LDS, by one wave.
T2V_DEV void rows64_dma(float* lds, const float* g, int row0, int L, int lane) {
  const int r = min(row0 + lane, L - 1);
  __builtin_amdgcn_global_load_lds(g + r, (lds_void*)lds, 4, 0, 0);
}

// ------------------------------------------------------------------- backward: dK, dV

// One 32-query step for this wave's 32 keys. RAGGED: only the first nvalid queries of
// the step are inside the clip (their P is forced to zero).
template <int D, bool RAGGED>
T2V_DEV void dkdv_step(uint32_t qbase, uint32_t gbase, uint32_t qr0, uint32_t qr1, uint32_t gr0, uint32_t gr1,
                       const float* sL2, const float* sDl, int qs, int nvalid,
                       float c, const bf16x8 (&kop)[D / 16], const bf16x8 (&vop)[D / 16], f32x16 (&dka)[D / 32],
                       f32x16 (&dva)[D / 32], int lane) {
  // Let the scheduler interleave this step's LDS reads with its MFMAs (measured: +2 to +4%).
  __builtin_amdgcn_iglp_opt(0);
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  const int l32 = lane & 31;
  // S and dP (32 queries x 32 keys): lane = key, register r = query qs + 8 (r/4) + 4 G + r % 4.
  bf16x8 aq[KK], ag[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) aq[kk] = read_opnd<D>(qbase, qs, kk);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) ag[kk] = read_opnd<D>(gbase, qs, kk);
  f32x16 s = zero16(), dp = zero16();
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) s = mfma(aq[kk], kop[kk], s);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) dp = mfma(ag[kk], vop[kk], dp);
  f32x4 lv[4], dl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lv[i] = *reinterpret_cast<const f32x4*>(sL2 + qs + i * 8 + G * 4);
    dl[i] = *reinterpret_cast<const f32x4*>(sDl + qs + i * 8 + G * 4);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float p = __builtin_amdgcn_exp2f(fmaf(s[r], c, -lv[r >> 2][r & 3]));
    if constexpr (RAGGED) {
      const int qi = (r >> 2) * 8 + G * 4 + (r & 3);
      p = qi < nvalid ? p : 0.0f;
    }
    s[r] = p;
    dp[r] = p * (dp[r] - dl[r >> 2][r & 3]);
  }
  const bf16x8 pb[2] = {to_bf16x8(s, 0), to_bf16x8(s, 8)};
  const bf16x8 sb[2] = {to_bf16x8(dp, 0), to_bf16x8(dp, 8)};
  // dV += P^T dO and dK += dS^T Q, contracting over the 16 queries of half hf.
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    bf16x8 bg[DB], bq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      bg[db] = read_rows_opnd<D>(gr0, gr1, qs + hf * 16, db);
      bq[db] = read_rows_opnd<D>(qr0, qr1, qs + hf * 16, db);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      dva[db] = mfma(pb[hf], bg[db], dva[db]);
      dka[db] = mfma(sb[hf], bq[db], dka[db]);
    }
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, 1) void attn_bwd_dkdv_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ delta,
    const Item* __restrict__ items, int H, int64_t T, float c, float scale, bf16* __restrict__ dk,
    bf16* __restrict__ dv) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  constexpr int BM = kDkdvBM;  // queries per LDS stage
  __shared__ __attribute__((aligned(1024))) bf16 sQ[2][BM * D];
  __shared__ __attribute__((aligned(1024))) bf16 sG[2][BM * D];  // dO
  __shared__ __attribute__((aligned(16))) float sL[2][BM];       // lse * log2(e)
  __shared__ __attribute__((aligned(16))) float sD[2][BM];       // Delta

  const Item it = items[blockIdx.x];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int G = lane >> 5;
  const int l32 = lane & 31;
  const int L = it.len;
  const int64_t rs = static_cast<int64_t>(H) * D;
  const int64_t base = static_cast<int64_t>(it.row0) * rs + static_cast<int64_t>(it.head) * D;
  const int64_t lbase = static_cast<int64_t>(it.head) * T + it.row0;
  const bf16* qh = q + base;
  const bf16* gh = dout + base;
  const float* l2h = lse2 + lbase;
  const float* dlh = delta + lbase;
  const int key_wave0 = it.tile0 + wave * 32;
  const bool wave_active = key_wave0 < L;

  auto stage = [&](int b, int i0) {
    tile_dma<D, BM, kThreads>(sQ[b], qh, rs, i0, L, tid);
    tile_dma<D, BM, kThreads>(sG[b], gh, rs, i0, L, tid);
    // BM floats of lse2 and of Delta, 64 per wave instruction (lanes past BM idle).
#pragma unroll
    for (int j = wave; j < 2 * ((BM + 63) / 64); j += kThreads / 64) {
      const int half = (BM + 63) / 64;
      const int part = j < half ? j : j - half;
      if (part * 64 + lane < BM)
        rows64_dma((j < half ? sL[b] : sD[b]) + part * 64, j < half ? l2h : dlh, i0 + part * 64, L, lane);
    }
  };
  stage(0, 0);

  // K and V of this wave's 32 keys, as B operands (lane = key, elements along head dim).
  bf16x8 kop[KK], vop[KK];
  {
    const int kj = key_wave0 + l32;
    const bool ok = kj < L;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kop[kk] = load8(k + base + kj * rs + kk * 16 + G * 8, ok);
      vop[kk] = load8(v + base + kj * rs + kk * 16 + G * 8, ok);
    }
  }
  f32x16 dka[DB], dva[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dka[db] = zero16();
    dva[db] = zero16();
  }

  const int ntiles = (L + BM - 1) / BM;
  const int nfull = L / BM;
  const uint32_t oo = opnd_lane_off<D>(lane);
  const uint32_t ro0 = rows_lane_off<D>(lane, 0), ro1 = rows_lane_off<D>(lane, 1);
  wait_vmcnt0();
  __syncthreads();
  for (int tt = 0; tt < nfull; ++tt) {
    const int b = tt & 1;
    if (tt + 1 < ntiles) stage(b ^ 1, (tt + 1) * BM);
    if (wave_active) {
      const uint32_t tq = lds_addr(sQ[b]), tg = lds_addr(sG[b]);
      const uint32_t qb = tq + oo, gb = tg + oo;
      const uint32_t q0 = tq + ro0, q1 = tq + ro1, g0 = tg + ro0, g1 = tg + ro1;
#pragma unroll
      for (int qs = 0; qs < BM; qs += 32)
        dkdv_step<D, false>(qb, gb, q0, q1, g0, g1, sL[b], sD[b], qs, 32, c, kop, vop, dka, dva, lane);
    }
    wait_vmcnt0();
    __syncthreads();
  }
  if (nfull < ntiles && wave_active) {  // last tile, 1 .. BM-1 queries
    const int b = nfull & 1;
    const int rem = L - nfull * BM;
    const uint32_t tq = lds_addr(sQ[b]), tg = lds_addr(sG[b]);
    const uint32_t qb = tq + oo, gb = tg + oo;
    const uint32_t q0 = tq + ro0, q1 = tq + ro1, g0 = tg + ro0, g1 = tg + ro1;
#pragma unroll
    for (int qs = 0; qs < BM; qs += 32) {
      if (rem >= qs + 32)
        dkdv_step<D, false>(qb, gb, q0, q1, g0, g1, sL[b], sD[b], qs, 32, c, kop, vop, dka, dva, lane);
      else if (rem > qs)
        dkdv_step<D, true>(qb, gb, q0, q1, g0, g1, sL[b], sD[b], qs, rem - qs, c, kop, vop, dka, dva, lane);
    }
  }

  if (wave_active) {
    // Accumulators: lane = head-dim column db*32 + l32, register r = key 8 (r/4) + 4 G + r % 4.
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int kj = key_wave0 + (r >> 2) * 8 + G * 4 + (r & 3);
      if (kj < L) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dk[base + kj * rs + db * 32 + l32] = static_cast<bf16>(dka[db][r] * scale);
          dv[base + kj * rs + db * 32 + l32] = static_cast<bf16>(dva[db][r]);
        }
      }
    }
  }
}

}  // namespace

int dkdv_tile_rows(int) { return (kThreads / 64) * 32; }

hipError_t launch_bwd_dkdv(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream) {
  const float c = a.scale * kLog2e;
  const dim3 grid(n_items), block(kThreads);
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  const auto* g = static_cast<const bf16*>(a.dout);
  auto* dk = static_cast<bf16*>(a.dk);
  auto* dv = static_cast<bf16*>(a.dv);
  const float* lse2 = a.delta + a.total_tokens * a.heads;
  if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<128>), grid, block, 0, stream, q, k, v, g, lse2, a.delta, items,
                       a.heads, a.total_tokens, c, a.scale, dk, dv);
  else
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<64>), grid, block, 0, stream, q, k, v, g, lse2, a.delta, items,
                       a.heads, a.total_tokens, c, a.scale, dk, dv);
  return hipGetLastError();
}
}  // namespace t2v
