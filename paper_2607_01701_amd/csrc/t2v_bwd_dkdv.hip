// Backward dK/dV kernel: a workgroup owns 32 keys per wave of one (clip, head) and loops
// over the clip's queries (see t2v_fwd.hip for the shared design notes). At head_dim 128
// four waves (128 keys, one workgroup per CU: 502 VGPRs) stage 64-query tiles; at 64, eight
// waves (256 keys, two per SIMD) share 128-query tiles, so each staged Q / dO tile feeds
// twice the waves (measured: +1-1.5% per fwd+bwd step at D = 64, results bitwise equal).
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

constexpr int kDkdvBM = 64;     // queries per LDS stage (a multiple of 32)
constexpr int kDkdvStages = 4;  // LDS stages: up to 3 tiles of Q / dO in flight during one tile's work
// Threads, queries per LDS stage and keys per workgroup by head_dim (32 keys per wave; each
// wave stages one 32-float piece of lse2 or -Delta per stage, so 2 BM = 32 waves).
template <int D>
constexpr int dkdv_threads() { return D == 64 ? 512 : kThreads; }
template <int D>
constexpr int dkdv_bm() { return D == 64 ? 128 : kDkdvBM; }
template <int D>
constexpr int dkdv_keys() { return dkdv_threads<D>() / 64 * 32; }

// Asynchronous copy of consecutive floats into LDS, one per active lane of the calling
// wave: lane i copies row i0 + off + i, clamped to L - 1, to lds[i]. The tile's first row
// i0 must be inside the clip (i0 < L); off + i may run past it, so the clamp is taken
// relative to i0 and the offset stays in [0, L - 1 - i0].
T2V_DEV void rows64_dma(float* lds, const float* g, int i0, int off, int L, int lane) {
  const uint32_t r = static_cast<uint32_t>(min(off + lane, L - 1 - i0));
#if T2V_CHECKED
  if (!check_row(i0 + static_cast<int>(r), L)) {  // copy the segment's first row instead
    dma_lds4_s(g, 0u, static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)lds)));
    return;
  }
#endif
  dma_lds4_s(g + i0, r * 4, static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)lds)));
}

// ------------------------------------------------------------------- backward: dK, dV

// Score operands of one 32-query step: rows qs .. qs + 31 of the Q and dO tiles.
template <int D>
T2V_DEV void dkdv_read_scores(uint32_t qbase, uint32_t gbase, int qs, bf16x8 (&aq)[D / 16], bf16x8 (&ag)[D / 16]) {
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) aq[kk] = read_opnd<D>(qbase, qs, kk);
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) ag[kk] = read_opnd<D>(gbase, qs, kk);
}

// S and dP - Delta of one 32-query step for this wave's 32 keys (32 queries x 32 keys):
// lane = key, register r = query qs + 8 (r/4) + 4 G + r % 4. dp arrives holding -Delta of
// each query (the accumulator's initial value), so the product lands on dP - Delta.
template <int D>
T2V_DEV void dkdv_scores_mfma(const bf16x8 (&aq)[D / 16], const bf16x8 (&ag)[D / 16], const bf16x8 (&kop)[D / 16],
                              const bf16x8 (&vop)[D / 16], f32x16& s, f32x16& dp) {
  s = zero16();
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) s = mfma(aq[kk], kop[kk], s);
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) dp = mfma(ag[kk], vop[kk], dp);
}

// P = exp2(c S - lse2) and dS = P (dP - Delta) of one step (dp holds dP - Delta), in bf16
// by 16-query half.
// RAGGED: only the first nvalid queries of the step are inside the clip (their P is
// forced to zero).
template <bool RAGGED>
T2V_DEV void dkdv_softmax(f32x16 s, f32x16 dp, const float* sL2, const float* sDl, int qs, int nvalid, float c,
                          bf16x8 (&pb)[2], bf16x8 (&sb)[2], int lane) {
  const int G = lane >> 5;
  f32x4 lv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) lv[i] = *reinterpret_cast<const f32x4*>(sL2 + qs + i * 8 + G * 4);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float p = __builtin_amdgcn_exp2f(fmaf(s[r], c, -lv[r >> 2][r & 3]));
    if constexpr (RAGGED) {
      const int qi = (r >> 2) * 8 + G * 4 + (r & 3);
      p = qi < nvalid ? p : 0.0f;
    }
    s[r] = p;
    dp[r] = p * dp[r];
  }
  pb[0] = to_bf16x8(s, 0);
  pb[1] = to_bf16x8(s, 8);
  sb[0] = to_bf16x8(dp, 0);
  sb[1] = to_bf16x8(dp, 8);
}

// dV += P^T dO and dK += dS^T Q for one step, contracting over the 16 queries of each half.
// All dV products come first: they need only P, so the dS arithmetic finishes under them
// before the dK products need it (measured: dK/dV +1-2% against alternating the two).
template <int D>
T2V_DEV void dkdv_grad_mfma(const bf16x8 (&pb)[2], const bf16x8 (&sb)[2], uint32_t qr0, uint32_t qr1, uint32_t gr0,
                            uint32_t gr1, int qs, f32x16 (&dka)[D / 32], f32x16 (&dva)[D / 32]) {
  constexpr int DB = D / 32;
  bf16x8 bg[2][DB], bq[2][DB];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) bg[hf][db] = read_rows_opnd<D>(gr0, gr1, qs + hf * 16, db);
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) dva[db] = mfma(pb[hf], bg[hf][db], dva[db]);
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) bq[hf][db] = read_rows_opnd<D>(qr0, qr1, qs + hf * 16, db);
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) dka[db] = mfma(sb[hf], bq[hf][db], dka[db]);
}

// One 32-query step (full, or the masked last step of a clip).
template <int D, bool RAGGED>
T2V_DEV void dkdv_step(uint32_t qbase, uint32_t gbase, uint32_t qr0, uint32_t qr1, uint32_t gr0, uint32_t gr1,
                       const float* sL2, const float* sDl, int qs, int nvalid,
                       float c, const bf16x8 (&kop)[D / 16], const bf16x8 (&vop)[D / 16], f32x16 (&dka)[D / 32],
                       f32x16 (&dva)[D / 32], int lane) {
  // Let the scheduler interleave this step's LDS reads with its MFMAs (measured: +2 to +4%).
  __builtin_amdgcn_iglp_opt(0);
  bf16x8 aq[D / 16], ag[D / 16], pb[2], sb[2];
  f32x16 s, dp;
  {  // dP's accumulator starts at -Delta (stored negated by the preprocess)
    const int G = lane >> 5;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(sDl + qs + i * 8 + G * 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) dp[i * 4 + e] = x[e];
    }
  }
  dkdv_read_scores<D>(qbase, gbase, qs, aq, ag);
  dkdv_scores_mfma<D>(aq, ag, kop, vop, s, dp);
  dkdv_softmax<RAGGED>(s, dp, sL2, sDl, qs, nvalid, c, pb, sb, lane);
  dkdv_grad_mfma<D>(pb, sb, qr0, qr1, gr0, gr1, qs, dka, dva);
}

template <int D, bool PERSIST>
__global__ __launch_bounds__(dkdv_threads<D>(), 1) void attn_bwd_dkdv_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ ndelta,
    const Item* __restrict__ items, int H, int64_t T, float c, float scale, bf16* __restrict__ dk,
    bf16* __restrict__ dv, float* __restrict__ partial, unsigned long long* __restrict__ trace, int n_items) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  constexpr int BM = dkdv_bm<D>();  // queries per LDS stage
  constexpr int NS = kDkdvStages;  // LDS stages in flight
  constexpr int NW = dkdv_threads<D>() / 64;
  // DMA instructions per wave and stage: the Q and dO tiles, plus one 32-float piece of
  // lse * log2(e) or -Delta.
  constexpr int kOps = 2 * (BM * D / 512) / NW + 1;
  static_assert(2 * BM == 32 * NW, "each wave stages one 32-float piece of lse2 / -Delta");
  __shared__ __attribute__((aligned(1024))) bf16 sQ[NS][BM * D];
  __shared__ __attribute__((aligned(1024))) bf16 sG[NS][BM * D];  // dO
  __shared__ __attribute__((aligned(16))) float sL[NS][BM];       // lse * log2(e)
  __shared__ __attribute__((aligned(16))) float sD[NS][BM];       // -Delta

  // One work item per workgroup, or (persistent grid) items w, w + grid, w + 2 grid, ...: the
  // grid is a multiple of the 8 XCDs, so every item still runs on XCD (item mod 8).
  for (int w = blockIdx.x, first = 1; PERSIST ? w < n_items : first != 0; w += gridDim.x, first = 0) {
    const unsigned long long trace_t0 = trace != nullptr ? trace_clock() : 0ull;
    const Item it = items[w];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = lane >> 5;
    const int l32 = lane & 31;
    const int Lk = it.len;   // keys of the sequence (this tile's rows)
    const int L = it.llen;   // queries of the sequence (the loop)
    const int64_t rs = static_cast<int64_t>(H) * D;
    const int64_t base = static_cast<int64_t>(it.row0) * rs + static_cast<int64_t>(it.head) * D;
    const int64_t qbase = static_cast<int64_t>(it.lrow0) * rs + static_cast<int64_t>(it.head) * D;
    const int64_t lbase = static_cast<int64_t>(it.head) * T + it.lrow0;
    const bf16* qh = q + qbase;
    const bf16* gh = dout + qbase;
    const float* vec_src = (wave < NW / 2 ? lse2 : ndelta) + lbase;
    const int vec_off = (wave % (NW / 2)) * 32;
    const int key_wave0 = it.tile0 + wave * 32;
    const bool wave_active = key_wave0 < Lk;

    // Every wave issues exactly kOps DMA instructions per stage, so counted waits work.
    const TileDma<D, BM, dkdv_threads<D>()> dma(tid, rs);
    auto stage = [&](int t) {
      const int b = t % NS, i0 = t * BM;
      dma.copy(sQ[b], qh, rs, i0, L);
      dma.copy(sG[b], gh, rs, i0, L);
      float* dst = (wave < NW / 2 ? sL[b] : sD[b]) + vec_off;
      if (lane < 32) rows64_dma(dst, vec_src, i0, vec_off, L, lane);
    };
    // Before reading stage t + 1: wait for it, leaving the stages issued after it in flight.
    auto wait_next = [&](int t, int ntiles) {
      const int after = min(NS - 2, ntiles - 2 - t);  // stages issued after t + 1
      if (after >= NS - 2) {
        wait_vmcnt<(NS - 2) * kOps>();
      } else if (NS > 3 && after == 1) {
        wait_vmcnt<kOps>();
      } else if (NS > 4 && after == 2) {
        wait_vmcnt<2 * kOps>();
      } else {
        wait_vmcnt0();
      }
    };
    static_assert(NS >= 2 && NS <= 5, "wait_next handles up to 3 stages in flight");

    const int ntiles = (L + BM - 1) / BM;
    const int nfull = L / BM;
    stage(0);

    // K and V of this wave's 32 keys, as B operands (lane = key, elements along head dim).
    bf16x8 kop[KK], vop[KK];
    {
      const int kj = key_wave0 + l32;
      const bool ok = kj < Lk;
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
    // Stage 0 and the K / V loads complete here; a wait the compiler sees also keeps it
    // from waiting for the K / V loads inside the loop (where the stages it does not see
    // would make that a full wait).
    wait_vmcnt0();
  #pragma unroll
    for (int t = 1; t < NS - 1; ++t)
      if (t < ntiles) stage(t);
    __syncthreads();

    const uint32_t oo = opnd_lane_off<D>(lane);
    const uint32_t ro0 = rows_lane_off<D>(lane, 0), ro1 = rows_lane_off<D>(lane, 1);
    for (int tt = 0; tt < nfull; ++tt) {
      const int b = tt % NS;
      if (tt + NS - 1 < ntiles) stage(tt + NS - 1);
      if (wave_active) {
        const uint32_t tq = lds_addr(sQ[b]), tg = lds_addr(sG[b]);
        const uint32_t qb = tq + oo, gb = tg + oo;
        const uint32_t q0 = tq + ro0, q1 = tq + ro1, g0 = tg + ro0, g1 = tg + ro1;
  #pragma unroll
        for (int qs = 0; qs < BM; qs += 32)
          dkdv_step<D, false>(qb, gb, q0, q1, g0, g1, sL[b], sD[b], qs, 32, c, kop, vop, dka, dva, lane);
      }
      wait_next(tt, ntiles);
      __syncthreads();
    }
    if (nfull < ntiles && wave_active) {  // last tile, 1 .. BM-1 queries
      const int b = nfull % NS;
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

    if (wave_active && it.slot >= 0) {
      // One piece of a split loop: unscaled fp32 sums into the item's partial slot
      // ([dK | dV] x tile key x head dim), added up in piece order by the reduce kernel.
      float* pk = partial + static_cast<int64_t>(it.slot) * (2 * dkdv_keys<D>() * D);
      float* pv = pk + dkdv_keys<D>() * D;
  #pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kr = wave * 32 + (r >> 2) * 8 + G * 4 + (r & 3);  // key within the tile
        if (it.tile0 + kr < Lk) {
  #pragma unroll
          for (int db = 0; db < DB; ++db) {
            pk[kr * D + db * 32 + l32] = dka[db][r];
            pv[kr * D + db * 32 + l32] = dva[db][r];
          }
        }
      }
    } else if (wave_active) {
      // Accumulators: lane = head-dim column db*32 + l32, register r = key 8 (r/4) + 4 G + r % 4.
  #pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int kj = key_wave0 + (r >> 2) * 8 + G * 4 + (r & 3);
        if (kj < Lk) {
  #pragma unroll
          for (int db = 0; db < DB; ++db) {
            dk[base + kj * rs + db * 32 + l32] = static_cast<bf16>(dka[db][r] * scale);
            dv[base + kj * rs + db * 32 + l32] = static_cast<bf16>(dva[db][r]);
          }
        }
      }
    }
    if (trace != nullptr) trace_end(trace, trace_t0, 2, w);
    if constexpr (PERSIST) {
      if (w + static_cast<int>(gridDim.x) < n_items) __syncthreads();  // LDS reads done before the next item's DMA
    }
  }
}

// Sum of the partial slots of one split tile, in piece order, scaled (dK) and rounded to
// bf16. A workgroup takes 32 keys of a tile; each thread four consecutive head-dim columns.
template <int D>
__global__ __launch_bounds__(kThreads) void dkdv_reduce_kernel(const float* __restrict__ partial,
                                                               const Item* __restrict__ tiles, int H, float scale,
                                                               bf16* __restrict__ dk, bf16* __restrict__ dv) {
  constexpr int kQuarters = dkdv_keys<D>() / 32;
  constexpr int C4 = D / 4;  // float4 columns per key row
  const Item it = tiles[blockIdx.x / kQuarters];
  const int k0 = (blockIdx.x % kQuarters) * 32;  // first key of this block, within the tile
  const int nkeys = min(32, it.len - it.tile0 - k0);
  const int64_t rs = static_cast<int64_t>(H) * D;
  const int64_t slot_elems = 2 * dkdv_keys<D>() * D;
  for (int e = threadIdx.x; e < 2 * 32 * C4; e += kThreads) {
    const int which = e / (32 * C4);  // 0: dK, 1: dV
    const int r = (e / C4) % 32;
    const int c4 = e % C4;
    if (r >= nkeys) continue;
    const float* src = partial + static_cast<int64_t>(it.slot) * slot_elems + which * dkdv_keys<D>() * D +
                       (k0 + r) * D + c4 * 4;
    f32x4 acc = *reinterpret_cast<const f32x4*>(src);
    for (int p = 1; p < it.pieces; ++p) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(src + p * slot_elems);
      acc[0] += x[0];
      acc[1] += x[1];
      acc[2] += x[2];
      acc[3] += x[3];
    }
    const float m = which == 0 ? scale : 1.0f;
    bf16x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = static_cast<bf16>(acc[i] * m);
    bf16* dst = (which == 0 ? dk : dv) + static_cast<int64_t>(it.row0 + it.tile0 + k0 + r) * rs +
                static_cast<int64_t>(it.head) * D + c4 * 4;
    *reinterpret_cast<bf16x4*>(dst) = w;
  }
}

}  // namespace

int dkdv_tile_rows(int head_dim) { return head_dim == 64 ? dkdv_keys<64>() : dkdv_keys<128>(); }

int64_t dkdv_partial_slot_bytes(int head_dim) { return 2LL * dkdv_tile_rows(head_dim) * head_dim * 4; }

hipError_t launch_bwd_dkdv_reduce(const AttnArgs& a, const Item* tiles, int n_tiles, hipStream_t stream) {
  const dim3 grid(n_tiles * (dkdv_tile_rows(a.head_dim) / 32)), block(kThreads);
  auto* dk = static_cast<bf16*>(a.dk);
  auto* dv = static_cast<bf16*>(a.dv);
  if (a.head_dim == 128)
    hipLaunchKernelGGL((dkdv_reduce_kernel<128>), grid, block, 0, stream, a.partial, tiles, a.heads, a.scale, dk, dv);
  else
    hipLaunchKernelGGL((dkdv_reduce_kernel<64>), grid, block, 0, stream, a.partial, tiles, a.heads, a.scale, dk, dv);
  return hipGetLastError();
}

namespace {
template <int D>
void launch_dkdv_as(const AttnArgs& a, const bf16* q, const bf16* k, const bf16* v, const bf16* g, const float* lse2,
                    const Item* items, int n_items, float c, bf16* dk, bf16* dv, hipStream_t stream) {
  const dim3 block(dkdv_threads<D>());
  if (a.persistent) {
    const void* fn = reinterpret_cast<const void*>(&attn_bwd_dkdv_kernel<D, true>);
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, true>), dim3(persistent_grid(fn, dkdv_threads<D>(), n_items)), block,
                       0, stream, q, k, v, g, lse2, a.delta, items, a.heads, a.total_tokens, c, a.scale, dk, dv,
                       a.partial, a.trace, n_items);
  } else {
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, false>), dim3(n_items), block, 0, stream, q, k, v, g, lse2, a.delta,
                       items, a.heads, a.total_tokens, c, a.scale, dk, dv, a.partial, a.trace, n_items);
  }
}
}  // namespace

hipError_t launch_bwd_dkdv(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream) {
  const float c = a.scale * kLog2e;
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  const auto* g = static_cast<const bf16*>(a.dout);
  auto* dk = static_cast<bf16*>(a.dk);
  auto* dv = static_cast<bf16*>(a.dv);
  const float* lse2 = a.delta + a.total_tokens * a.heads;
  if (a.head_dim == 128)
    launch_dkdv_as<128>(a, q, k, v, g, lse2, items, n_items, c, dk, dv, stream);
  else
    launch_dkdv_as<64>(a, q, k, v, g, lse2, items, n_items, c, dk, dv, stream);
  return hipGetLastError();
}
#if T2V_CHECKED
hipError_t dkdv_check_take(unsigned int* rec, unsigned int canary) { return kern::check_take_here(rec, canary); }
#endif
}  // namespace t2v
