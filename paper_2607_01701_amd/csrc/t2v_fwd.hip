// gfx950 kernels for packed variable-length bidirectional attention.
//
// One workgroup processes one work item (a tile of one clip and one head, from the host
// scheduler): 8 waves / 256 queries (or 4 waves / 128 queries for short key segments) in
// the forward and dQ kernels, 4 waves / 128 keys in the dK/dV kernel. All products use v_mfma_f32_32x32x16_bf16 with fp32 accumulation;
// K/V (forward, dQ) or Q/dO (dK/dV) tiles are staged through LDS ahead of use (two
// buffers in the forward and dQ kernels, four in dK/dV), one barrier per tile.
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
// dK/dV kernel (a workgroup owns 128 keys, loops over the clip's queries, or over one
// piece of them when the host splits long loops) and a dQ kernel (a workgroup owns a
// query tile, loops over the clip's keys). P is recomputed from the stored lse; split
// loops leave fp32 partial sums that a reduce kernel adds in a fixed order, so there are
// no atomics and results are bitwise reproducible.
#include "t2v_kernel_common.hpp"

namespace t2v {

using namespace kern;

namespace {

constexpr int kFwdQB = 1;  // 32-query blocks per wave
constexpr int kFwdBN = 64; // keys per LDS stage (a multiple of 32)
// Wide tiles: eight waves (two per SIMD, 256 queries) share each staged K/V tile, so every
// tile crosses from L2 into LDS once per 256 queries rather than once per 128 (measured:
// forward +3-5% against two independent 4-wave workgroups per CU on long clips). Narrow
// tiles: four waves (128 queries), two workgroups per CU, for packs whose key segments are
// short: there one workgroup's Q loads and O stores overlap the other's MFMA work.
constexpr int kFwdThreadsWide = 512;
constexpr int kFwdThreadsNarrow = 256;

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
T2V_DEV float ext(float a, float b) {
  return NEG ? min_nan(a, b) : max_nan(a, b);
}

template <bool NEG>
T2V_DEV float tree_ext16(const f32x16& x) {
  float a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = ext<NEG>(x[i], x[i + 8]);
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = ext<NEG>(a[i], a[i + 4]);
  return ext<NEG>(ext<NEG>(a[0], a[2]), ext<NEG>(a[1], a[3]));
}

// One 32-key step of the forward pass for QB query blocks of this wave.
// sK/sV: the LDS stage; kb: first key of the step within the stage; nvalid: keys of the
// step inside the clip (only read when RAGGED, where it is 1..31).
template <int D, int QB, bool NEG, bool RAGGED>
T2V_DEV void fwd_step(uint32_t kbase, uint32_t vbase0, uint32_t vbase1, int kb, int nvalid, float c,
                      const bf16x8 (&qop)[QB][D / 16], f32x16 (&o)[QB][D / 32], float (&m_run)[QB],
                      float (&l_run)[QB], int lane) {
  // Let the scheduler interleave this step's LDS reads with its MFMAs (measured: +2 to +4%).
  __builtin_amdgcn_iglp_opt(0);
  constexpr int KK = D / 16;
  constexpr int DB = D / 32;
  const int G = lane >> 5;
  // S^T (32 keys x 32 queries per block): lane = query, register r = key 8 (r/4) + 4 G + r % 4.
  bf16x8 ka[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) ka[kk] = read_opnd<D>(kbase, kb, kk);
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
    for (int db = 0; db < DB; ++db) va[hf][db] = read_rows_opnd<D>(vbase0, vbase1, kb + hf * 16, db);
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

template <int D, int QB, bool NEG, int NT, bool PERSIST>
__global__ __launch_bounds__(NT, 512 / NT) void attn_fwd_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ k, const bf16* __restrict__ v,
    const Item* __restrict__ items, int H, int64_t T, float c, bf16* __restrict__ out,
    float* __restrict__ lse, unsigned long long* __restrict__ trace, int n_items) {
  constexpr int KK = D / 16;  // k-steps of the head-dim contraction
  constexpr int DB = D / 32;  // 32-wide head-dim blocks of the output
  constexpr int BN = kFwdBN;  // keys per LDS stage
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
    const int64_t rs = static_cast<int64_t>(H) * D;  // elements between consecutive tokens
    const int64_t base = static_cast<int64_t>(it.row0) * rs + static_cast<int64_t>(it.head) * D;
    const int64_t kvbase = static_cast<int64_t>(it.lrow0) * rs + static_cast<int64_t>(it.head) * D;
    const bf16* kh = k + kvbase;
    const bf16* vh = v + kvbase;
    const int q_wave0 = it.tile0 + wave * QB * 32;
    const bool wave_active = q_wave0 < Lq;

    const TileDma<D, BN, NT> dma(tid, rs);
    dma.copy(sK[0], kh, rs, 0, L);
    dma.copy(sV[0], vh, rs, 0, L);

    bf16x8 qop[QB][KK];
  #pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int qi = q_wave0 + qb * 32 + l32;
      const bool ok = qi < Lq;
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
    const int nfull = L / BN;  // tiles with BN keys of the sequence
    const uint32_t ko = opnd_lane_off<D>(lane);
    const uint32_t vo0 = rows_lane_off<D>(lane, 0), vo1 = rows_lane_off<D>(lane, 1);
    wait_vmcnt0();
    __syncthreads();
    for (int tt = 0; tt < nfull; ++tt) {
      const int b = tt & 1;
      if (tt + 1 < ntiles) {
        dma.copy(sK[b ^ 1], kh, rs, (tt + 1) * BN, L);
        dma.copy(sV[b ^ 1], vh, rs, (tt + 1) * BN, L);
      }
      if (wave_active) {
        const uint32_t kbase = lds_addr(sK[b]) + ko;
        const uint32_t vb0 = lds_addr(sV[b]) + vo0, vb1 = lds_addr(sV[b]) + vo1;
  #pragma unroll
        for (int kb = 0; kb < BN; kb += 32)
          fwd_step<D, QB, NEG, false>(kbase, vb0, vb1, kb, 32, c, qop, o, m_run, l_run, lane);
      }
      wait_vmcnt0();
      __syncthreads();
    }
    if (nfull < ntiles && wave_active) {  // last tile, 1 .. BN-1 keys
      const int b = nfull & 1;
      const int rem = L - nfull * BN;
      const uint32_t kbase = lds_addr(sK[b]) + ko;
      const uint32_t vb0 = lds_addr(sV[b]) + vo0, vb1 = lds_addr(sV[b]) + vo1;
  #pragma unroll
      for (int kb = 0; kb < BN; kb += 32) {
        if (rem >= kb + 32)
          fwd_step<D, QB, NEG, false>(kbase, vb0, vb1, kb, 32, c, qop, o, m_run, l_run, lane);
        else if (rem > kb)
          fwd_step<D, QB, NEG, true>(kbase, vb0, vb1, kb, rem - kb, c, qop, o, m_run, l_run, lane);
      }
    }

    if (wave_active) {
  #pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int qi = q_wave0 + qb * 32 + l32;
        const float lt = half_sum(l_run[qb]);
        const float inv = 1.0f / lt;
        if (qi < Lq) {
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
    if (trace != nullptr) trace_end(trace, trace_t0, 0, w);
    if constexpr (PERSIST) {
      if (w + static_cast<int>(gridDim.x) < n_items) __syncthreads();  // LDS reads done before the next item's DMA
    }
  }
}

}  // namespace

int fwd_tile_rows(int, bool narrow) { return ((narrow ? kFwdThreadsNarrow : kFwdThreadsWide) / 64) * 32 * kFwdQB; }

namespace {
template <int D, bool NEG, int NT>
void launch_fwd_as(const AttnArgs& a, const bf16* q, const bf16* k, const bf16* v, bf16* o, float* lse,
                   const Item* items, int n_items, float c, hipStream_t stream) {
  if (a.persistent) {
    const void* fn = reinterpret_cast<const void*>(&attn_fwd_kernel<D, kFwdQB, NEG, NT, true>);
    hipLaunchKernelGGL((attn_fwd_kernel<D, kFwdQB, NEG, NT, true>), dim3(persistent_grid(fn, NT, n_items)), dim3(NT),
                       0, stream, q, k, v, items, a.heads, a.total_tokens, c, o, lse, a.trace, n_items);
  } else {
    hipLaunchKernelGGL((attn_fwd_kernel<D, kFwdQB, NEG, NT, false>), dim3(n_items), dim3(NT), 0, stream, q, k, v,
                       items, a.heads, a.total_tokens, c, o, lse, a.trace, n_items);
  }
}

template <int D, bool NEG>
void launch_fwd_d(const AttnArgs& a, const bf16* q, const bf16* k, const bf16* v, bf16* o, float* lse,
                  const Item* items, int n_items, float c, hipStream_t stream) {
  if (a.q_rows == fwd_tile_rows(D, true))
    launch_fwd_as<D, NEG, kFwdThreadsNarrow>(a, q, k, v, o, lse, items, n_items, c, stream);
  else
    launch_fwd_as<D, NEG, kFwdThreadsWide>(a, q, k, v, o, lse, items, n_items, c, stream);
}
}  // namespace

hipError_t launch_fwd(const AttnArgs& a, void* out, float* lse, const Item* items, int n_items,
                      hipStream_t stream) {
  if (a.q_rows != fwd_tile_rows(a.head_dim, true) && a.q_rows != fwd_tile_rows(a.head_dim, false))
    return hipErrorInvalidValue;
  const float c = a.scale * kLog2e;
  const auto* q = static_cast<const bf16*>(a.q);
  const auto* k = static_cast<const bf16*>(a.k);
  const auto* v = static_cast<const bf16*>(a.v);
  auto* o = static_cast<bf16*>(out);
  const bool neg = a.scale < 0.0f;
  if (a.head_dim == 128) {
    if (neg)
      launch_fwd_d<128, true>(a, q, k, v, o, lse, items, n_items, c, stream);
    else
      launch_fwd_d<128, false>(a, q, k, v, o, lse, items, n_items, c, stream);
  } else {
    if (neg)
      launch_fwd_d<64, true>(a, q, k, v, o, lse, items, n_items, c, stream);
    else
      launch_fwd_d<64, false>(a, q, k, v, o, lse, items, n_items, c, stream);
  }
  return hipGetLastError();
}
#if T2V_CHECKED
hipError_t fwd_check_take(unsigned int* rec, unsigned int canary) { return kern::check_take_here(rec, canary); }
#endif
}  // namespace t2v
