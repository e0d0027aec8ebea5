// Shared constants of the gfx950 attention kernels (one workgroup = 4 waves, one work item).
#pragma once

#include "t2v_device.hpp"
#include "t2v_kernels.h"

namespace t2v {
namespace kern {


constexpr int kThreads = 256;  // 4 waves
constexpr float kTau = 8.0f;   // lazy-rescale threshold, log2 units

constexpr float kInf = __builtin_huge_valf();

}  // namespace kern
}  // namespace t2v
