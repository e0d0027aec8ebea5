// Launch interface between the C ABI (t2v_api.hip) and the kernels (t2v_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "t2v_host.h"

namespace t2v {

// Rows per work item of each kernel (the tile sizes the scheduler cuts clips into). The
// forward and dQ kernels come in a wide (8-wave) and a narrow (4-wave) form.
int fwd_tile_rows(int head_dim, bool narrow);
int dkdv_tile_rows(int head_dim);
int dq_tile_rows(int head_dim, bool narrow);
// Bytes of one dK/dV partial slot (fp32 dK and dV of one tile of keys).
int64_t dkdv_partial_slot_bytes(int head_dim);

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
  int q_rows = 0;            // forward / dQ tile rows: selects the wide or narrow kernels
  float* partial = nullptr;  // dK/dV partial slots of split loops (work items with slot >= 0)
  // Persistent grid: launch only as many workgroups as the GPU holds at once (a multiple of
  // the 8 XCDs), each taking items w, w + grid, ...; otherwise one workgroup per item.
  bool persistent = false;
};

// Workgroups of a persistent launch of `kernel` with `threads` threads: the resident
// workgroups per CU times the CUs, rounded down to a multiple of the XCD count, at most
// n_items (and at least 1).
int persistent_grid(const void* kernel, int threads, int n_items);

hipError_t launch_fwd(const AttnArgs& a, void* out, float* lse, const Item* items, int n_items,
                      hipStream_t stream);
hipError_t launch_bwd_pre(const AttnArgs& a, hipStream_t stream);
hipError_t launch_bwd_dkdv(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream);
hipError_t launch_bwd_dkdv_reduce(const AttnArgs& a, const Item* tiles, int n_tiles, hipStream_t stream);
hipError_t launch_bwd_dq(const AttnArgs& a, const Item* items, int n_items, hipStream_t stream);

#if T2V_CHECKED
// Checked builds only: the DMA row record of the forward, dK/dV and dQ kernel sources
// ({violations, first violating workgroup, its row, the segment length}); each call clears
// the record and sets the canary (rows taken off every bound) for the next launches.
hipError_t fwd_check_take(unsigned int* rec, unsigned int canary);
hipError_t dkdv_check_take(unsigned int* rec, unsigned int canary);
hipError_t dq_check_take(unsigned int* rec, unsigned int canary);
#endif

}  // namespace t2v
