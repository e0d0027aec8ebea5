// Host-side pieces of libt2vattn that need no HIP: argument validation, the tile
// scheduler and the thread-local error message. Compiled into the GPU library and,
// alone, into a host-only library with g++ for CPU tests.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace t2v {

// One unit of kernel work: a tile of `block` rows of one (sequence, head). A kernel owns
// the tile's rows (queries in the forward and dQ kernels, keys in the dK/dV kernel) and
// loops over the sequence's other segment (its keys, or its queries). For self-attention
// both segments are the clip itself.
struct Item {
  int32_t row0;   // first row of the owned segment in its packed tensor
  int32_t len;    // owned segment length
  int32_t tile0;  // first row of the tile, relative to row0
  int32_t head;   // head index
  int32_t lrow0;  // first row of the looped-over segment in its packed tensor
  int32_t llen;   // looped-over segment length (>= 1 whenever len >= 1)
  int32_t pad0, pad1;
};
static_assert(sizeof(Item) == 32, "Item is one 256-bit scalar load");

constexpr int kNumXcd = 8;  // MI355X: 8 accelerator dies; workgroups are dealt round-robin

// Thread-local last-error text; set_error returns the status it is given.
int set_error(int status, const std::string& msg);
const char* last_error();

// Validates the shape arguments shared by forward and backward. On success stores T
// (total tokens) and returns T2V_OK; otherwise returns the status and sets the error.
int validate_shape(const int32_t* cu, int nseq, int heads, int head_dim, float scale, int64_t* total_tokens);

// Pointer checks: non-null, 16-byte aligned, and the byte ranges given do not overlap.
struct Range {
  const void* ptr;
  int64_t bytes;
  const char* name;
};
int validate_pointers(const std::vector<Range>& inputs, const std::vector<Range>& outputs);

// Validates separate query / key offsets: both as validate_shape (same nseq), and every
// sequence has either both queries and keys or neither. Stores Tq and Tk.
int validate_shape_qk(const int32_t* cu_q, const int32_t* cu_k, int nseq, int heads, int head_dim, float scale,
                      int64_t* tq, int64_t* tk);

// Builds the work list for tiles of `block` rows of the owned segments (offsets cu_own),
// each looping over the matching segment of cu_loop (see t2v_build_worklist in t2vattn.h;
// self-attention passes the same offsets twice).
std::vector<Item> build_worklist(const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads, int block,
                                 int order);

// Greedy list-scheduling makespan of `items` on `slots` workers, dealt per XCD when
// slots is a multiple of kNumXcd. Costs are tile rows x looped-over length.
void plan_makespan(const Item* items, int n, int block, int slots, double* makespan, double* lower_bound);

}  // namespace t2v
