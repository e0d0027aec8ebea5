// Device helpers for the gfx950 (CDNA4) attention kernels: vector types, the bf16
// 32x32x16 MFMA, LDS operand reads (plain and transposing) and cross-lane helpers.
//
// MFMA v_mfma_f32_32x32x16_bf16 lane layout (wave64, l = lane, G = l / 32, t = 0..7):
//   A[m][k]: lane l holds m = l % 32, k = 8 G + t          (8 bf16 per lane)
//   B[k][n]: lane l holds k = 8 G + t, n = l % 32           (8 bf16 per lane)
//   C[m][n]: lane l, register r holds m = 8 (r / 4) + 4 G + (r % 4), n = l % 32  (16 fp32)
// The contraction index k only has to agree between A and B, so every product below
// chooses its own assignment of keys/queries to (G, t).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace t2v {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#define T2V_DEV __device__ __forceinline__

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

T2V_DEV f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

T2V_DEV f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

T2V_DEV bf16x8 zero_bf16x8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

// 16-byte global load of 8 bf16; returns zeros when !valid (the address is not touched).
T2V_DEV bf16x8 load8(const bf16* p, bool valid) {
  if (valid) return *reinterpret_cast<const bf16x8*>(p);
  return zero_bf16x8();
}

T2V_DEV u32x4 load_raw16(const bf16* p, bool valid) {
  if (valid) return *reinterpret_cast<const u32x4*>(p);
  u32x4 z = {0u, 0u, 0u, 0u};
  return z;
}

// 16-byte LDS read (ds_read_b128).
T2V_DEV bf16x8 lds_read8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// ds_read_b64_tr_b16: within each group of 16 lanes, source lane s supplies the address
// of 4 consecutive bf16; output lane j receives, as element c, element (j % 4) of source
// lane 4c + j / 4. With source lane s pointing at row (base + s / 4), column (cb + 4 (s % 4))
// of a row-major tile, output lane j gets rows base + 0..3 of column cb + j.
T2V_DEV bf16x4 lds_read_tr4(const bf16* p) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  return __builtin_bit_cast(bf16x4, v);
}

// MFMA operand whose contraction index runs down the rows of a row-major LDS tile
// (rows = keys or queries, columns = head dim): element t of lane l is
// tile[row0 + 8 (t / 4) + 4 G + (t % 4)][col0 + l % 32]. Two transposing reads.
T2V_DEV bf16x8 lds_read_rows_operand(const bf16* tile, int stride, int row0, int col0, int lane) {
  const int G = lane >> 5;
  const int s = lane & 15;
  const int dhalf = (lane >> 4) & 1;
  const bf16* p = tile + (row0 + 4 * G + (s >> 2)) * stride + col0 + 16 * dhalf + 4 * (s & 3);
  bf16x4 lo = lds_read_tr4(p);
  bf16x4 hi = lds_read_tr4(p + 8 * stride);
  bf16x8 r;
  r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
  r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
  return r;
}

// ---------------------------------------------------------------- swizzled LDS tiles
//
// A tile of R rows x D bf16 is stored unpadded (row stride D) with its 16-byte chunks
// permuted within each row: logical chunk c of row r sits in slot c ^ swz<D>(r). gfx950's
// LDS serves 256 bytes (64 banks of 4 bytes) per cycle, i.e. 16 lanes of a 16-byte read.
// For D = 128 (256-byte rows) swz permutes r mod 16 onto 0..15 so that both access patterns
// are free of bank conflicts: sixteen consecutive rows at one chunk (the 16-byte operand
// reads) and four consecutive rows x two adjacent chunks per 16 lanes (the transposing 8-byte
// reads); measured 186 and 93 bytes/clock/CU, against 100 and 92 for an 8-way permutation.
// For D = 64 (128-byte rows, two rows per bank line) it permutes (r / 2) mod 8.
template <int D>
T2V_DEV int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  return (r >> 1) & 7;
}

// Element offset of (row r, column col) in a swizzled tile; col % 8 is kept.
template <int D>
T2V_DEV int swz_off(int r, int col) {
  return r * D + (((col >> 3) ^ swz<D>(r)) << 3) + (col & 7);
}

typedef __attribute__((address_space(3))) void lds_void;

// A wave-uniform pointer, moved to SGPRs (a no-op when the compiler already keeps it there).
T2V_DEV const void* uniform_ptr(const void* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
  return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// LDS DMA (global_load_lds) of 16 or 4 bytes per lane from sbase + voff: a wave-uniform
// 64-bit base in SGPRs plus a per-lane 32-bit byte offset, so a tile's addresses cost no
// 64-bit vector math. Lane i writes LDS bytes [lds + W i, lds + W (i + 1)), W = 16 or 4;
// `lds` must be wave-uniform (it goes to M0).
//
// Written as inline assembly on purpose: for the compiler's builtin form, the wait-count
// pass cannot tell which LDS bytes a DMA writes, so it puts a full vmcnt(0) wait before
// the next LDS read, which makes every prefetch finish before the current tile's work
// starts. Here the compiler does not see the DMA at all, and the kernels order it
// themselves with counted vmcnt waits before the barrier that publishes a stage. (The
// compiler's own waits for ordinary loads stay correct: unseen DMAs only make them wait
// longer.) The compiler does not look inside the assembly for hazards either: the s_nop
// gives the 5 wait states a vector memory instruction needs after a VALU write of an SGPR
// it reads (the base may come from v_readfirstlane), which also covers the M0 write.
T2V_DEV void dma_lds16_s(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(uniform_ptr(sbase)), "{m0}"(lds)
               : "memory");
}
T2V_DEV void dma_lds4_s(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(uniform_ptr(sbase)), "{m0}"(lds)
               : "memory");
}

// ---------------------------------------------------------------------- checked builds
//
// Compiled with T2V_CHECKED=1 (the separate checked library), every DMA checks that the row
// it copies lies inside its segment (the clip, or the piece of it a work item loops over).
// Each kernel source file keeps one record per device, {violations, workgroup, row, bound,
// canary}; the host clears it before a call and reads it after the call's kernels finish.
// The canary (set by the host on request) shortens every bound by that many rows, so correct
// kernels report their segments' last rows; the copies themselves are unchanged. A row that
// fails the check is not copied: the DMA reads the segment's first row instead, keeping every
// wave's count of DMA instructions (and so the counted waits) as in the unchecked kernels.
#ifndef T2V_CHECKED
#define T2V_CHECKED 0
#endif
#if T2V_CHECKED
static __device__ unsigned int t2v_check_rec[5];

// True when 0 <= row < bound - canary; otherwise counts a violation and keeps the first.
T2V_DEV bool check_row(int row, int bound) {
  const int b = bound - static_cast<int>(t2v_check_rec[4]);
  if (row >= 0 && row < b) return true;
  if (atomicAdd(&t2v_check_rec[0], 1u) == 0u) {
    t2v_check_rec[1] = blockIdx.x;
    t2v_check_rec[2] = static_cast<unsigned int>(row);
    t2v_check_rec[3] = static_cast<unsigned int>(bound);
  }
  return false;
}
#endif

// Asynchronous copy of rows row0 .. row0 + R - 1 of one (clip, head) into a swizzled LDS
// tile with global_load_lds_dwordx4 (each wave instruction fills 1 KB of LDS; lane i the
// 16 bytes at offset 16 i). Rows at or past `L` are replaced by row L - 1, so the tile only
// ever holds finite input values; callers mask those rows. Each wave issues
// R * D / 512 / (NTHREADS / 64) DMA instructions; completion must be awaited with a vmcnt
// wait before a barrier that precedes reads of the tile.
//
// Wave w's instruction j covers tile rows RPI (w + NW j) .. + RPI - 1. The swizzle depends
// on the row modulo 16 and RPI * NW is a multiple of 16, so a lane's chunk is the same for
// every j and its byte offset is one per-lane constant plus a wave-uniform j * RPI * NW * rs;
// only the clip's last, partial tile needs per-lane clamping.
template <int D, int R, int NTHREADS>
struct TileDma {
  static constexpr int CPR = D / 8;     // chunks per row
  static constexpr int RPI = 64 / CPR;  // rows per wave instruction
  static constexpr int NI = R / RPI;    // wave instructions per tile
  static constexpr int NW = NTHREADS / 64;
  static constexpr int NJ = NI / NW;    // instructions per wave
  static_assert(R % RPI == 0 && NI % NW == 0, "tile shape must fill whole wave instructions");
  static_assert((RPI * NW) % 16 == 0, "a lane's swizzled chunk must not depend on the instruction");
  int wave;       // uniform
  int r0;         // this lane's row in instruction 0
  uint32_t col;   // byte offset of its 16-byte chunk within the row
  uint32_t off0;  // r0 * row bytes + col

  T2V_DEV TileDma(int tid, int64_t rs) {
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    r0 = RPI * wave + lane / CPR;
    col = static_cast<uint32_t>(((lane % CPR) ^ swz<D>(r0)) * 16);
    off0 = static_cast<uint32_t>(r0) * static_cast<uint32_t>(rs * 2) + col;
  }

  // g: token 0 of the clip for this head; rs: token stride in elements.
  T2V_DEV void copy(bf16* tile, const bf16* g, int64_t rs, int row0, int L) const {
    const char* base = reinterpret_cast<const char*>(g + static_cast<int64_t>(row0) * rs);
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)tile)) + wave * 1024;
    const int64_t step = static_cast<int64_t>(RPI * NW) * rs * 2;  // bytes between instructions
    if (row0 + R <= L) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#if T2V_CHECKED
        if (!check_row(row0 + r0 + RPI * NW * j, L)) {
          dma_lds16_s(g, col, lds0 + j * NW * 1024);
          continue;
        }
#endif
        dma_lds16_s(base + j * step, off0, lds0 + j * NW * 1024);
      }
    } else {
      const int last = L - 1 - row0;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int r = min(r0 + RPI * NW * j, last);
#if T2V_CHECKED
        if (!check_row(row0 + r, L)) {
          dma_lds16_s(g, col, lds0 + j * NW * 1024);
          continue;
        }
#endif
        dma_lds16_s(base, static_cast<uint32_t>(r) * static_cast<uint32_t>(rs * 2) + col, lds0 + j * NW * 1024);
      }
    }
  }
};

// Waits until this thread's outstanding vector memory operations (including LDS DMA) are done.
T2V_DEV void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Waits until at most N of this thread's vector memory operations are outstanding. They
// complete in issue order, so this waits for everything issued before the last N.
template <int N>
T2V_DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit field");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte operand read of logical chunk `chunk` of row r from a swizzled tile.
template <int D>
T2V_DEV bf16x8 swz_read8(const bf16* tile, int r, int chunk) {
  return *reinterpret_cast<const bf16x8*>(tile + r * D + ((chunk ^ swz<D>(r)) << 3));
}

// As lds_read_rows_operand, for a swizzled tile with row stride D.
template <int D>
T2V_DEV bf16x8 swz_read_rows_operand(const bf16* tile, int row0, int col0, int lane) {
  const int G = lane >> 5;
  const int s = lane & 15;
  const int dhalf = (lane >> 4) & 1;
  const int r = row0 + 4 * G + (s >> 2);
  const int col = col0 + 16 * dhalf + 4 * (s & 3);
  bf16x4 lo = lds_read_tr4(tile + swz_off<D>(r, col));
  bf16x4 hi = lds_read_tr4(tile + swz_off<D>(r + 8, col));
  bf16x8 out;
  out[0] = lo[0]; out[1] = lo[1]; out[2] = lo[2]; out[3] = lo[3];
  out[4] = hi[0]; out[5] = hi[1]; out[6] = hi[2]; out[7] = hi[3];
  return out;
}

// ---------------------------------------------------------------- LDS addressing
//
// Operand reads address swizzled tiles with 32-bit LDS byte addresses. Two identities
// (checked exhaustively for every lane on the host, see tests/test_lds_layout.py) make each read one
// base register plus one XOR: for the 16-byte operand of row (32j + lane % 32), chunk 2 kk + G,
//   off(kk) = off(0) ^ (kk << 5) ;
// for the transposing read of rows (16i + 4G + s/4 + 8h), column 32 db + 16 dh + 4 (s % 4),
//   off(db) = off(0) ^ (db << 6) ;
// and rows that differ by a multiple of 16 differ by a constant (folded into the instruction's
// immediate offset). Tile bases are 1 KB aligned, so base + (o ^ x) == (base + o) ^ x.
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

T2V_DEV uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_char*)p));
}
T2V_DEV bf16x8 lds_ld8(uint32_t a) { return *(const lds_bf16x8*)(a); }
T2V_DEV bf16x4 lds_ld_tr4(uint32_t a) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(a)));
}

// Byte offsets of this lane's reads within a swizzled tile (row base 0, kk = 0, db = 0).
template <int D>
T2V_DEV uint32_t opnd_lane_off(int lane) {
  return 2u * static_cast<uint32_t>(swz_off<D>(lane & 31, 8 * (lane >> 5)));
}
template <int D>
T2V_DEV uint32_t rows_lane_off(int lane, int h) {
  const int G = lane >> 5, s = lane & 15, dh = (lane >> 4) & 1;
  return 2u * static_cast<uint32_t>(swz_off<D>(4 * G + (s >> 2) + 8 * h, 16 * dh + 4 * (s & 3)));
}

// 16-byte operand: row row0 + lane % 32 (row0 a multiple of 32), chunk 2 kk + G.
template <int D>
T2V_DEV bf16x8 read_opnd(uint32_t base, int row0, int kk) {
  return lds_ld8((base ^ static_cast<uint32_t>(kk << 5)) + static_cast<uint32_t>(row0 * 2 * D));
}

// Operand whose contraction index runs down the rows (see lds_read_rows_operand), rows
// row0 .. row0 + 15 (row0 a multiple of 16), columns 32 db .. 32 db + 31.
template <int D>
T2V_DEV bf16x8 read_rows_opnd(uint32_t base0, uint32_t base1, int row0, int db) {
  const uint32_t x = static_cast<uint32_t>(db << 6), ro = static_cast<uint32_t>(row0 * 2 * D);
  const bf16x4 lo = lds_ld_tr4((base0 ^ x) + ro);
  const bf16x4 hi = lds_ld_tr4((base1 ^ x) + ro);
  bf16x8 out;
  out[0] = lo[0]; out[1] = lo[1]; out[2] = lo[2]; out[3] = lo[3];
  out[4] = hi[0]; out[5] = hi[1]; out[6] = hi[2]; out[7] = hi[3];
  return out;
}

// ---------------------------------------------------------------- workgroup trace
//
// Measurement only. When a launch is traced, each workgroup writes one record of four
// uint64 at rec + 4 * blockIdx.x: the CU it ran on ((XCC_ID << 16) | HW_ID bits 8..15,
// i.e. CU, shader array and shader engine within the XCD), its start and end on the
// constant 100 MHz clock, and the kernel's slot.
T2V_DEV unsigned long long trace_clock() { return __builtin_amdgcn_s_memrealtime(); }

// Every wave of the workgroup must call this (it holds a barrier); rec is uniform. `index` is the
// work item's position in the list (the record written).
T2V_DEV void trace_end(unsigned long long* rec, unsigned long long t0, int slot, int index) {
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned hw, xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const unsigned long long t1 = __builtin_amdgcn_s_memrealtime();
    unsigned long long* r = rec + 4 * static_cast<size_t>(index);
    r[0] = (static_cast<unsigned long long>(xcc & 0xFu) << 16) | ((hw >> 8) & 0xFFu);
    r[1] = t0;
    r[2] = t1;
    r[3] = static_cast<unsigned long long>(slot);
  }
}

// Eight fp32 to packed bf16 (round to nearest even, v_cvt_pk_bf16_f32).
T2V_DEV bf16x8 to_bf16x8(const f32x16& x, int base) {
  bf16x8 r;
#pragma unroll
  for (int t = 0; t < 8; ++t) r[t] = static_cast<bf16>(x[base + t]);
  return r;
}

// v_permlane32_swap with both operands x: element 0 then holds x from lane l % 32 and
// element 1 holds x from lane 32 + l % 32, in every lane. These combine a value with
// its partner in the other half of the wave (lane l ^ 32).
T2V_DEV float half_sum(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

// NaN-propagating maximum / minimum (v_maximum3_f32 / v_minimum3_f32 on gfx950). Unlike
// fmaxf / fminf they need no canonicalising copies of operands that come straight from an
// MFMA, and a NaN score carries through to a NaN output instead of being dropped.
T2V_DEV float max_nan(float a, float b) { return __builtin_elementwise_maximum(a, b); }
T2V_DEV float min_nan(float a, float b) { return __builtin_elementwise_minimum(a, b); }

T2V_DEV float half_max(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return max_nan(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

T2V_DEV float half_min(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return min_nan(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

}  // namespace t2v
