// gfx950 kernels for packed variable-length bidirectional attention.
//
// One workgroup = 4 waves = 256 threads, one work item (a tile of one clip and one
// head, from the host scheduler). All products use v_mfma_f32_32x32x16_bf16 with fp32
// accumulation; K/V (forward, dQ) or Q/dO (dK/dV) tiles are staged through LDS with a
// two-buffer pipeline: the global loads for tile t+1 are issued before the MFMA work on
// tile t and land in the other LDS buffer after it, one barrier per tile.
//
// Forward (paper Section III, Observation 2: full self-attention over each clip):
// every lane owns one query row of a 32-query block, because scores are computed
// transposed (S^T = K Q^T), so row max/sum need one swap with the other wave half.
// The softmax is online over 32-key steps with a lazily moved reference maximum:
// the reference m only moves when a step's maximum exceeds it by more than kTau (in
// log2 units), which keeps every exp2 argument <= kTau and lets most steps skip the
// rescale of the output accumulator. The final O / l and lse = ln2 (m + log2 l) are
// exact for any reference m, so the result is the plain softmax up to rounding.
//
// Backward (Fig. 1 caption: the DiT backward pass): Delta = rowsum(dO * O), then a
// dK/dV kernel (a workgroup owns 128 keys, loops over the clip's queries) and a dQ
// kernel (a workgroup owns a query tile, loops over the clip's keys). P is recomputed
// from the stored lse; nothing is accumulated across workgroups, so there are no
// atomics and results are bitwise reproducible.
#include "t2v_device.hpp"
#include "t2v_kernels.h"

namespace t2v {

namespace {

constexpr int kThreads = 256;  // 4 waves
constexpr float kTau = 8.0f;   // lazy-rescale threshold, log2 units
constexpr int kFwdQB = 1;      // 32-query blocks per wave, forward
constexpr int kDqQB = 1;       // 32-query blocks per wave, dQ

constexpr float kInf = __builtin_huge_valf();

// ------------------------------------------------------------------------------ forward

// Sum / max of the 16 values of an accumulator as a balanced tree (short dependency chains).
T2V_DEV float tree_sum16(const f32x16& x) {
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = x[i] + x[i + 8];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] += a[i + 4];
  return (a[0] + a[2]) + (a[1] + a[3]);
}

template <bool NEG>
T2V_DEV float tree_ext16(const f32x16& x) {
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = NEG ? fminf(x[i], x[i + 8]) : fmaxf(x[i], x[i + 8]);
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = NEG ? fminf(a[i], a[i + 4]) : fmaxf(a[i], a[i + 4]);
  const float b0 = NEG ? fminf(a[0], a[2]) : fmaxf(a[0], a[2]);
  const float b1 = NEG ? fminf(a[1], a[3]) : fmaxf(a[1], a[3]);
  return NEG ? fminf(b0, b1) : fmaxf(b0, b1);
}

// One 32-key step of the forward pass for QB query blocks of this wave.
// sK/sV: the LDS stage; kb: first key of the step within the stage; nvalid: keys of the
// step inside the clip (only read when RAGGED, where it is 1..31).
template <int D, int QB, bool NEG, bool RAGGED>
T2V_DEV void fwd_step(const bf16* sK, const bf16* sV, int kb, int nvalid, float c,
                      const bf16x8 (&qop)[QB][D / 16], f32x16 (&o)[QB][D / 32], float (&m_run)[QB],
                      float (&l_run)[QB], int lane) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  const int l32 = lane & 31;
  // S^T (32 keys x 32 queries per block): lane = query, register r = key 8 (r/4) + 4 G + r % 4.
  bf16x8 ka[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) ka[kk] = swz_read8<D>(sK, kb + l32, 2 * kk + G);
  f32x16 s[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) s[qb] = zero16();
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) s[qb] = mfma(ka[kk], qop[qb][kk], s[qb]);
  }
  // V operands are read now so their LDS latency overlaps the softmax arithmetic.
  bf16x8 va[2][DB];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) va[hf][db] = swz_read_rows_operand<D>(sV, kb + hf * 16, db * 32, lane);
  bf16x8 pb[QB][2];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    if constexpr (RAGGED) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = (r >> 2) * 8 + G * 4 + (r & 3);
        if (key >= nvalid) s[qb][r] = NEG ? kInf : -kInf;
      }
    }
    float mx = tree_ext16<NEG>(s[qb]);
    mx = NEG ? half_min(mx) : half_max(mx);
    const float mblk = mx * c;  // largest scaled score of this step
    if (__any(mblk > m_run[qb] + kTau)) {
      const float mn = fmaxf(m_run[qb], mblk);
      const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - mn);
      l_run[qb] *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[qb][db] *= alpha;
      m_run[qb] = mn;
    }
    const float nm = -m_run[qb];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float p = __builtin_amdgcn_exp2f(fmaf(s[qb][r], c, nm));
      if constexpr (RAGGED) {
        const int key = (r >> 2) * 8 + G * 4 + (r & 3);
        p = key < nvalid ? p : 0.0f;  // also covers scale = 0, where c * -inf is NaN
      }
      s[qb][r] = p;
    }
    l_run[qb] += tree_sum16(s[qb]);
    pb[qb][0] = to_bf16x8(s[qb], 0);
    pb[qb][1] = to_bf16x8(s[qb], 8);
  }
  // O^T += V^T P^T: the key of P element t (from register 8 hf + t) is
  // kb + 16 hf + 8 (t / 4) + 4 G + t % 4, which is how the V operand is read.
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) o[qb][db] = mfma(va[hf][db], pb[qb][hf], o[qb][db]);
    }
  }
}

template <int D, int QB, bool NEG>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const Item* __restrict__ items, int H, int64_t T, float c, bf16* __restrict__ out,
    float* __restrict__ lse) {
  constexpr int KK = D / 16;  // k-steps of the head-dim contraction
  constexpr int DB = D / 32;  // 32-wide head-dim blocks of the output
  constexpr int BN = 64;      // keys per LDS stage
  __shared__ __attribute__((aligned(1024))) bf16 sK[2][BN * D];
  __shared__ __attribute__((aligned(1024))) bf16 sV[2][BN * D];

  const Item it = items[blockIdx.x];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int G = lane >> 5;
  const int l32 = lane & 31;
  const int L = it.len;
  const int64_t rs = static_cast<int64_t>(H) * D;  // elements between consecutive tokens
  const int64_t base = static_cast<int64_t>(it.row0) * rs + static_cast<int64_t>(it.head) * D;
  const bf16* kh = k + base;
  const bf16* vh = v + base;
  const int q_wave0 = it.tile0 + wave * QB * 32;
  const bool wave_active = q_wave0 < L;

  tile_dma<D, BN, kThreads>(sK[0], kh, rs, 0, L, tid);
  tile_dma<D, BN, kThreads>(sV[0], vh, rs, 0, L, tid);

  bf16x8 qop[QB][KK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qi = q_wave0 + qb * 32 + l32;
    const bool ok = qi < L;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qop[qb][kk] = load8(q + base + qi * rs + kk * 16 + G * 8, ok);
  }

  f32x16 o[QB][DB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -kInf;
    l_run[qb] = 0.0f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[qb][db] = zero16();
  }

  const int ntiles = (L + BN - 1) / BN;
  const int nfull = L / BN;  // tiles with BN keys of the clip
  wait_vmcnt0();
  __syncthreads();
  for (int tt = 0; tt < nfull; ++tt) {
    const int b = tt & 1;
    if (tt + 1 < ntiles) {
      tile_dma<D, BN, kThreads>(sK[b ^ 1], kh, rs, (tt + 1) * BN, L, tid);
      tile_dma<D, BN, kThreads>(sV[b ^ 1], vh, rs, (tt + 1) * BN, L, tid);
    }
    if (wave_active) {
      fwd_step<D, QB, NEG, false>(sK[b], sV[b], 0, 32, c, qop, o, m_run, l_run, lane);
      fwd_step<D, QB, NEG, false>(sK[b], sV[b], 32, 32, c, qop, o, m_run, l_run, lane);
    }
    wait_vmcnt0();
    __syncthreads();
  }
  if (nfull < ntiles && wave_active) {  // last tile, 1 .. BN-1 keys
    const int b = nfull & 1;
    const int rem = L - nfull * BN;
    if (rem >= 32) {
      fwd_step<D, QB, NEG, false>(sK[b], sV[b], 0, 32, c, qop, o, m_run, l_run, lane);
      if (rem > 32) fwd_step<D, QB, NEG, true>(sK[b], sV[b], 32, rem - 32, c, qop, o, m_run, l_run, lane);
    } else {
      fwd_step<D, QB, NEG, true>(sK[b], sV[b], 0, rem, c, qop, o, m_run, l_run, lane);
    }
  }

  if (wave_active) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qi = q_wave0 + qb * 32 + l32;
      const float lt = half_sum(l_run[qb]);
      const float inv = 1.0f / lt;
      if (qi < L) {
        bf16* orow = out + base + qi * rs;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            bf16x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = static_cast<bf16>(o[qb][db][i * 4 + e] * inv);
            *reinterpret_cast<bf16x4*>(orow + db * 32 + i * 8 + G * 4) = w;
          }
        }
        if (G == 0) lse[static_cast<int64_t>(it.head) * T + it.row0 + qi] = (m_run[qb] + __builtin_amdgcn_logf(lt)) * kLn2;
      }
    }
  }
}

// ------------------------------------------------------------------- backward: Delta

// Delta[h, t] = sum_d dO[t, h, d] O[t, h, d]  and  lse2[h, t] = lse[h, t] * log2(e).
template <int D>
__global__ __launch_bounds__(kThreads) void attn_bwd_pre_kernel(const bf16* __restrict__ out,
                                                                 const bf16* __restrict__ dout,
                                                                 const float* __restrict__ lse, int64_t rows,
                                                                 int H, int64_t T, float* __restrict__ delta,
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
      delta[h * T + t] = acc;
      lse2[h * T + t] = lse[h * T + t] * kLog2e;
    }
  }
}

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
T2V_DEV void dkdv_step(const bf16* sQ, const bf16* sG, const float* sL2, const float* sDl, int qs, int nvalid,
                       float c, const bf16x8 (&kop)[D / 16], const bf16x8 (&vop)[D / 16], f32x16 (&dka)[D / 32],
                       f32x16 (&dva)[D / 32], int lane) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  const int l32 = lane & 31;
  // S and dP (32 queries x 32 keys): lane = key, register r = query qs + 8 (r/4) + 4 G + r % 4.
  bf16x8 aq[KK], ag[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) aq[kk] = swz_read8<D>(sQ, qs + l32, 2 * kk + G);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) ag[kk] = swz_read8<D>(sG, qs + l32, 2 * kk + G);
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
      bg[db] = swz_read_rows_operand<D>(sG, qs + hf * 16, db * 32, lane);
      bq[db] = swz_read_rows_operand<D>(sQ, qs + hf * 16, db * 32, lane);
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
  constexpr int BM = 64;  // queries per LDS stage
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
    if (wave == 0) rows64_dma(sL[b], l2h, i0, L, lane);
    if (wave == 1) rows64_dma(sD[b], dlh, i0, L, lane);
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
  wait_vmcnt0();
  __syncthreads();
  for (int tt = 0; tt < nfull; ++tt) {
    const int b = tt & 1;
    if (tt + 1 < ntiles) stage(b ^ 1, (tt + 1) * BM);
    if (wave_active) {
      dkdv_step<D, false>(sQ[b], sG[b], sL[b], sD[b], 0, 32, c, kop, vop, dka, dva, lane);
      dkdv_step<D, false>(sQ[b], sG[b], sL[b], sD[b], 32, 32, c, kop, vop, dka, dva, lane);
    }
    wait_vmcnt0();
    __syncthreads();
  }
  if (nfull < ntiles && wave_active) {  // last tile, 1 .. BM-1 queries
    const int b = nfull & 1;
    const int rem = L - nfull * BM;
    if (rem >= 32) {
      dkdv_step<D, false>(sQ[b], sG[b], sL[b], sD[b], 0, 32, c, kop, vop, dka, dva, lane);
      if (rem > 32) dkdv_step<D, true>(sQ[b], sG[b], sL[b], sD[b], 32, rem - 32, c, kop, vop, dka, dva, lane);
    } else {
      dkdv_step<D, true>(sQ[b], sG[b], sL[b], sD[b], 0, rem, c, kop, vop, dka, dva, lane);
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

// ------------------------------------------------------------------------ backward: dQ

// One 32-key step for this wave's QB query blocks. RAGGED: only the first nvalid keys of
// the step are inside the clip.
template <int D, int QB, bool RAGGED>
T2V_DEV void dq_step(const bf16* sK, const bf16* sV, int kb, int nvalid, float c, const bf16x8 (&qop)[QB][D / 16],
                     const bf16x8 (&gop)[QB][D / 16], const float (&nl2)[QB], const float (&dlt)[QB],
                     f32x16 (&dqa)[QB][D / 32], int lane) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  const int l32 = lane & 31;
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
    for (int kk = 0; kk < KK; ++kk) ka[kk] = swz_read8<D>(sK, kb + l32, 2 * kk + G);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) s[qb] = mfma(ka[kk], qop[qb][kk], s[qb]);
  }
  {
    bf16x8 va[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) va[kk] = swz_read8<D>(sV, kb + l32, 2 * kk + G);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) dp[qb] = mfma(va[kk], gop[qb][kk], dp[qb]);
  }
  bf16x8 kt[2][DB];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int db = 0; db < DB; ++db) kt[hf][db] = swz_read_rows_operand<D>(sK, kb + hf * 16, db * 32, lane);
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
      s[qb][r] = p * (dp[qb][r] - dlt[qb]);
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

template <int D, int QB>
__global__ __launch_bounds__(kThreads, 2) void attn_bwd_dq_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const bf16* __restrict__ dout, const float* __restrict__ lse2, const float* __restrict__ delta,
    const Item* __restrict__ items, int H, int64_t T, float c, float scale, bf16* __restrict__ dq) {
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  constexpr int BN = 64;
  __shared__ __attribute__((aligned(1024))) bf16 sK[2][BN * D];
  __shared__ __attribute__((aligned(1024))) bf16 sV[2][BN * D];

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
  const bf16* kh = k + base;
  const bf16* vh = v + base;
  const int q_wave0 = it.tile0 + wave * QB * 32;
  const bool wave_active = q_wave0 < L;

  tile_dma<D, BN, kThreads>(sK[0], kh, rs, 0, L, tid);
  tile_dma<D, BN, kThreads>(sV[0], vh, rs, 0, L, tid);

  bf16x8 qop[QB][KK], gop[QB][KK];
  float nl2[QB], dlt[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qi = q_wave0 + qb * 32 + l32;
    const bool ok = qi < L;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qop[qb][kk] = load8(q + base + qi * rs + kk * 16 + G * 8, ok);
      gop[qb][kk] = load8(dout + base + qi * rs + kk * 16 + G * 8, ok);
    }
    nl2[qb] = ok ? -lse2[lbase + qi] : 0.0f;
    dlt[qb] = ok ? delta[lbase + qi] : 0.0f;
  }
  f32x16 dqa[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int db = 0; db < DB; ++db) dqa[qb][db] = zero16();

  const int ntiles = (L + BN - 1) / BN;
  const int nfull = L / BN;
  wait_vmcnt0();
  __syncthreads();
  for (int tt = 0; tt < nfull; ++tt) {
    const int b = tt & 1;
    if (tt + 1 < ntiles) {
      tile_dma<D, BN, kThreads>(sK[b ^ 1], kh, rs, (tt + 1) * BN, L, tid);
      tile_dma<D, BN, kThreads>(sV[b ^ 1], vh, rs, (tt + 1) * BN, L, tid);
    }
    if (wave_active) {
      dq_step<D, QB, false>(sK[b], sV[b], 0, 32, c, qop, gop, nl2, dlt, dqa, lane);
      dq_step<D, QB, false>(sK[b], sV[b], 32, 32, c, qop, gop, nl2, dlt, dqa, lane);
    }
    wait_vmcnt0();
    __syncthreads();
  }
  if (nfull < ntiles && wave_active) {
    const int b = nfull & 1;
    const int rem = L - nfull * BN;
    if (rem >= 32) {
      dq_step<D, QB, false>(sK[b], sV[b], 0, 32, c, qop, gop, nl2, dlt, dqa, lane);
      if (rem > 32) dq_step<D, QB, true>(sK[b], sV[b], 32, rem - 32, c, qop, gop, nl2, dlt, dqa, lane);
    } else {
      dq_step<D, QB, true>(sK[b], sV[b], 0, rem, c, qop, gop, nl2, dlt, dqa, lane);
    }
  }

  if (wave_active) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qi = q_wave0 + qb * 32 + l32;
      if (qi < L) {
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
}

}  // namespace

int fwd_tile_rows(int) { return (kThreads / 64) * 32 * kFwdQB; }
int dkdv_tile_rows(int) { return (kThreads / 64) * 32; }
int dq_tile_rows(int) { return (kThreads / 64) * 32 * kDqQB; }

hipError_t launch_fwd(const AttnArgs& a, void* out, float* lse, const Item* items, int n_items,
                      hipStream_t stream) {
  const float c = a.scale * kLog2e;
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  auto* o = static_cast<bf16*>(out);
  const dim3 grid(n_items), block(kThreads);
  const bool neg = a.scale < 0.0f;
  if (a.head_dim == 128) {
    if (neg)
      hipLaunchKernelGGL((attn_fwd_kernel<128, kFwdQB, true>), grid, block, 0, stream, q, k, v, items, a.heads,
                         a.total_tokens, c, o, lse);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<128, kFwdQB, false>), grid, block, 0, stream, q, k, v, items, a.heads,
                         a.total_tokens, c, o, lse);
  } else {
    if (neg)
      hipLaunchKernelGGL((attn_fwd_kernel<64, kFwdQB, true>), grid, block, 0, stream, q, k, v, items, a.heads,
                         a.total_tokens, c, o, lse);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<64, kFwdQB, false>), grid, block, 0, stream, q, k, v, items, a.heads,
                         a.total_tokens, c, o, lse);
  }
  return hipGetLastError();
}

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

hipError_t launch_bwd_dq(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream) {
  const float c = a.scale * kLog2e;
  const dim3 grid(n_items), block(kThreads);
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  const auto* g = static_cast<const bf16*>(a.dout);
  auto* dq = static_cast<bf16*>(a.dq);
  const float* lse2 = a.delta + a.total_tokens * a.heads;
  if (a.head_dim == 128)
    hipLaunchKernelGGL((attn_bwd_dq_kernel<128, kDqQB>), grid, block, 0, stream, q, k, v, g, lse2, a.delta,
                       items, a.heads, a.total_tokens, c, a.scale, dq);
  else
    hipLaunchKernelGGL((attn_bwd_dq_kernel<64, kDqQB>), grid, block, 0, stream, q, k, v, g, lse2, a.delta,
                       items, a.heads, a.total_tokens, c, a.scale, dq);
  return hipGetLastError();
}

}  // namespace t2v
