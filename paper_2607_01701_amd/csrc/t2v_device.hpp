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

T2V_DEV float half_max(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

T2V_DEV float half_min(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fminf(__builtin_bit_cast(float, (unsigned)r[0]), __builtin_bit_cast(float, (unsigned)r[1]));
}

}  // namespace t2v
