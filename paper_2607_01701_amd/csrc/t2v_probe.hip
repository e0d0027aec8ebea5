// MFMA throughput probe: the bf16 dense rate this chip sustains at the clock it holds under a
// pure v_mfma_f32_32x32x16_bf16 load. The attention kernels' rates are quoted against AMD's
// published peak; this probe gives the same chip's measured ceiling beside it, as context.
#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "../../include/t2vattn.h"
#include "t2v_device.hpp"
#include "t2v_host.h"

namespace t2v {
namespace {

constexpr int kProbeThreads = 256;  // one wave per SIMD
constexpr int kChains = 4;          // independent accumulators per wave

// Every wave runs kChains independent MFMA accumulation chains for `iters` rounds, with no
// memory traffic in the loop. Thread 0 of each workgroup writes its three record words
// (shader-clock ticks, wall-clock ticks, a checksum), so writes stay inside rec[3 * gridDim.x).
__global__ __launch_bounds__(kProbeThreads) void mfma_peak_kernel(int iters, unsigned long long* rec) {
  const unsigned t = threadIdx.x + 1u;
  u32x4 ua = {t, t * 3u, t * 5u, t * 7u}, ub = {t * 11u, t * 13u, t * 17u, t * 19u};
  // Small finite bf16 values (exponent bits masked), so the sums stay finite.
  ua &= 0x3C7F3C7Fu;
  ub &= 0x3C7F3C7Fu;
  const bf16x8 a = __builtin_bit_cast(bf16x8, ua), b = __builtin_bit_cast(bf16x8, ub);
  f32x16 acc[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) acc[j] = zero16();
  const long long c0 = clock64(), w0 = wall_clock64();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < kChains; ++j) acc[j] = mfma(a, b, acc[j]);
  }
  const long long c1 = clock64(), w1 = wall_clock64();
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < kChains; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  if (threadIdx.x == 0) {
    rec[3 * blockIdx.x] = static_cast<unsigned long long>(c1 - c0);
    rec[3 * blockIdx.x + 1] = static_cast<unsigned long long>(w1 - w0);
    rec[3 * blockIdx.x + 2] = static_cast<unsigned long long>(__builtin_bit_cast(unsigned, s));
  }
}

int fail(hipError_t e, const char* what) {
  return set_error(T2V_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

}  // namespace
}  // namespace t2v

extern "C" int t2v_probe_mfma_peak(unsigned long long* rec, int blocks, int iters, void* stream, double* ms_out,
                                   double* tflops_out, double* ghz_out) {
  using namespace t2v;
  if (rec == nullptr || ms_out == nullptr || tflops_out == nullptr || ghz_out == nullptr)
    return set_error(T2V_ERR_INVALID_ARG, "NULL argument");
  if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 24))
    return set_error(T2V_ERR_INVALID_ARG, "blocks must be in [1, 2^20] and iters in [1, 2^24]");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0, wall_khz = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev);
  if (e != hipSuccess) return fail(e, "device query");
  if (wall_khz <= 0) return set_error(T2V_ERR_HIP, "device reports no wall-clock rate");
  hipEvent_t ev[2] = {nullptr, nullptr};
  if ((e = hipEventCreate(&ev[0])) != hipSuccess || (e = hipEventCreate(&ev[1])) != hipSuccess) {
    if (ev[0] != nullptr) (void)hipEventDestroy(ev[0]);
    return fail(e, "hipEventCreate");
  }
  std::vector<unsigned long long> host(3 * static_cast<size_t>(blocks));
  float ms = 0.0f;
  e = hipEventRecord(ev[0], s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(kProbeThreads), 0, s, iters, rec);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(ev[1], s);
  if (e == hipSuccess) e = hipMemcpyAsync(host.data(), rec, host.size() * sizeof(unsigned long long),
                                          hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev[0], ev[1]);
  (void)hipEventDestroy(ev[0]);
  (void)hipEventDestroy(ev[1]);
  if (e != hipSuccess) return fail(e, "MFMA probe");
  double clk = 0.0, wall = 0.0;
  for (int i = 0; i < blocks; ++i) {
    clk += static_cast<double>(host[3 * i]);
    wall += static_cast<double>(host[3 * i + 1]);
  }
  const double flops = 32.0 * 32.0 * 16.0 * 2.0 * kChains * (kProbeThreads / 64) * static_cast<double>(iters) *
                       static_cast<double>(blocks);
  *ms_out = ms;
  *tflops_out = ms > 0.0f ? flops / (ms * 1e-3) * 1e-12 : 0.0;
  *ghz_out = wall > 0.0 ? clk / wall * (wall_khz * 1e-6) : 0.0;
  return T2V_OK;
}
