// Shared constants of the gfx950 attention kernels (one workgroup = 4 waves, one work item).
#pragma once

#include "t2v_device.hpp"
#include "t2v_kernels.h"

namespace t2v {
namespace kern {


constexpr int kThreads = 256;  // 4 waves
constexpr float kTau = 8.0f;   // lazy-rescale threshold, log2 units

constexpr float kInf = __builtin_huge_valf();

#if T2V_CHECKED
// Checked builds: copies this source file's DMA row record ({violations, workgroup, row,
// bound}) to `rec`, then clears it and sets the canary for the launches that follow. The
// copies are synchronous; the caller has waited for the kernels that wrote the record.
[[maybe_unused]] static hipError_t check_take_here(unsigned int* rec, unsigned int canary) {
  hipError_t e = hipMemcpyFromSymbol(rec, HIP_SYMBOL(t2v_check_rec), 4 * sizeof(unsigned int), 0,
                                     hipMemcpyDeviceToHost);
  if (e != hipSuccess) return e;
  const unsigned int fresh[5] = {0u, 0u, 0u, 0u, canary};
  return hipMemcpyToSymbol(HIP_SYMBOL(t2v_check_rec), fresh, sizeof(fresh), 0, hipMemcpyHostToDevice);
}
#endif

}  // namespace kern
}  // namespace t2v
