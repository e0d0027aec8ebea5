// Launch interface between the C ABI (t2v_api.hip) and the kernels (t2v_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "t2v_host.h"

namespace t2v {

// Rows per work item of each kernel (the tile sizes the scheduler cuts clips into).
int fwd_tile_rows(int head_dim);
int dkdv_tile_rows(int head_dim);
int dq_tile_rows(int head_dim);

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* out;   // forward output (written by fwd, read by bwd)
  const float* lse;  // [H, T]
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  float* delta;  // [2, H, T]: -Delta, then lse * log2(e)
  int heads;
  int head_dim;
  int64_t total_tokens;
  float scale;
  // Per-workgroup trace records of the launch being made (4 uint64 each), or nullptr.
  unsigned long long* trace = nullptr;
};

hipError_t launch_fwd(const AttnArgs& a, void* out, float* lse, const Item* items, int n_items,
                      hipStream_t stream);
hipError_t launch_bwd_pre(const AttnArgs& a, hipStream_t stream);
hipError_t launch_bwd_dkdv(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream);
hipError_t launch_bwd_dq(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream);

}  // namespace t2v
