// Host-side pieces of libt2vattn that need no HIP: argument validation, the tile
// scheduler and the thread-local error message. Compiled into the GPU library and,
// alone, into a host-only library with g++ for CPU tests.
#pragma once

#include <cstdint>
#include <string>
#include <utility>
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
  // Loop split (dK/dV only): when the looped-over segment is cut into `pieces` > 1 pieces,
  // the item covers one piece (lrow0 / llen describe the piece) and writes fp32 partial
  // sums to partial slot `slot`; otherwise slot = -1 and pieces = 1. In a reduce list the
  // item is one split tile, slot its first slot and pieces the slot count.
  int32_t slot;
  int32_t pieces;
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
// self-attention passes the same offsets twice). chunk > 0 cuts every looped-over segment
// longer than chunk rows into pieces (loop_pieces), one item per tile and piece; the
// partial slot of (sequence s, head h, tile t, piece j) is base(s, h) + t * pieces + j, with
// base counted over the split (sequence, head) pairs in pack order.
std::vector<Item> build_worklist(const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads, int block,
                                 int order, int chunk = 0);

// Pieces of a loop of LL rows cut at chunk rows: *n pieces of *step rows (a multiple of
// 64), the last taking the rest. *n = 1 (step = LL) when chunk <= 0 or LL <= chunk.
void loop_pieces(int LL, int chunk, int* n, int* step);

// Loop split of a work list (used for dK/dV, whose loop over a long query segment is the
// critical path when few key tiles exist, as in cross-attention against short text).
struct LoopSplit {
  int chunk = 0;       // rows per piece before rounding; 0: no split
  int64_t slots = 0;   // partial slots the pieces write
};
constexpr int kMinChunk = 2048;  // smallest piece: keeps the partial traffic small against the work

// No split unless the costliest tile (rows x loop length) exceeds an even share of all work
// over `parallel` workers; then pieces near an even share over 2 x parallel, at least
// kMinChunk rows, widened until the partial slots fit in max_slots.
LoopSplit choose_loop_split(const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads, int block,
                            int parallel, int64_t max_slots);

// Tile rows for a kernel that comes in a wide and a narrow form (the forward and dQ
// kernels: 256 or 128 query rows). Narrow when narrow_always, or when the work-weighted loop
// length sum(L L'^2) / sum(L L') is at most narrow_max_loop (owned length L, looped-over
// length L'); otherwise narrow only when the list-scheduling makespan of the narrow work list
// over `slots` workers, times narrow_penalty (the narrow kernel's measured cost per unit of
// work relative to the wide one on long loops), is below the wide list's: few tiles per CU
// leave the last round of wide tiles part-empty. When both lists were built for the
// comparison and `chosen` is given, the chosen one is moved into it (else it is left empty).
int choose_tile_rows(const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads, int wide, int narrow,
                     bool narrow_always, double narrow_max_loop, double narrow_penalty, int order, int slots,
                     std::vector<Item>* chosen = nullptr);

// One item per split tile of build_worklist(..., chunk): row0, len, tile0, head of the tile,
// slot = its first partial slot, pieces = the number of consecutive slots to sum.
std::vector<Item> build_reduce_list(const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads, int block,
                                    int chunk);

// Checks a kernel work list against the offsets it was built from (tile rows against
// cu_seqlens): each item's owned rows are one whole non-empty segment s of cu_own, its tile
// starts inside that segment at a multiple of `block`, its head is in [0, heads), and its
// looped-over rows lie inside segment s of cu_loop: all of it (slot = -1, pieces = 1), or one
// piece of it writing partial slot `slot` < max_slots (pieces >= 2). Items of a reduce list
// (reduce = true) have no loop; they need slots [slot, slot + pieces) below max_slots, with
// pieces >= 2. Returns an empty string for a valid list, else what is wrong with the first
// bad item. (Used by the checked library before a list reaches the GPU.)
std::string check_work_items(const Item* items, int n, const int32_t* cu_own, const int32_t* cu_loop, int nseq,
                             int heads, int block, int64_t max_slots, bool reduce);

// First-fit allocator of byte ranges inside one memory chunk of `size` bytes (host-side
// bookkeeping only: the chunk itself is device or pinned host memory owned by the caller).
// Sizes are rounded up to kAlign; freed neighbours coalesce.
class RangeAllocator {
 public:
  static constexpr uint64_t kAlign = 256;
  explicit RangeAllocator(uint64_t size = 0);
  uint64_t size() const { return size_; }
  // Offset of a free range of at least `bytes` (rounded up), or -1 when none is large enough.
  int64_t alloc(uint64_t bytes);
  // Returns a range obtained from alloc (same `bytes`); false if it is not a live range.
  bool release(uint64_t off, uint64_t bytes);
  uint64_t free_bytes() const { return free_total_; }
  size_t free_ranges() const { return free_.size(); }
  static uint64_t rounded(uint64_t bytes) { return (bytes + kAlign - 1) / kAlign * kAlign; }

 private:
  uint64_t size_ = 0, free_total_ = 0;
  std::vector<std::pair<uint64_t, uint64_t>> free_;  // (offset, length), sorted by offset, disjoint
};

// Greedy list-scheduling makespan of `items` on `slots` workers, dealt per XCD when
// slots is a multiple of kNumXcd. Costs are tile rows x looped-over length.
void plan_makespan(const Item* items, int n, int block, int slots, double* makespan, double* lower_bound);

}  // namespace t2v
