// Host-side validation and tile scheduling for libt2vattn (no HIP dependency).
//
// The scheduler mirrors, inside one GPU, the balance goal of the paper's planner:
// a clip's attention cost grows with L^2 (Eq. (9), alpha_2 * B * S^2), so a pack of
// clips of very different length (Section III, Observation 1; the 13- to 113-frame
// example of Fig. 1) leaves workers idle unless the longest work starts first. The
// planner's fitness function is a critical-path list scheduler; here every tile of a
// clip costs (tile rows x L) and the list is ordered longest clip first, which is
// greedy list scheduling in LPT order for the hardware's in-order dispatch.
#include "t2v_host.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <iterator>
#include <numeric>
#include <queue>

#include "../../include/t2vattn.h"

namespace t2v {

namespace {
thread_local std::string g_last_error;
}

int set_error(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

const char* last_error() { return g_last_error.c_str(); }

int validate_shape(const int32_t* cu, int nseq, int heads, int head_dim, float scale, int64_t* total_tokens) {
  if (nseq < 0) return set_error(T2V_ERR_INVALID_ARG, "nseq must be >= 0");
  if (cu == nullptr) return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (heads < 1) return set_error(T2V_ERR_INVALID_ARG, "heads must be >= 1");
  if (head_dim != 64 && head_dim != 128)
    return set_error(T2V_ERR_UNSUPPORTED, "head_dim must be 64 or 128, got " + std::to_string(head_dim));
  if (!std::isfinite(scale)) return set_error(T2V_ERR_INVALID_ARG, "scale must be finite");
  if (cu[0] != 0) return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  for (int s = 0; s < nseq; ++s) {
    if (cu[s + 1] < cu[s])
      return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens must be non-decreasing (index " + std::to_string(s + 1) + ")");
  }
  const int64_t T = cu[nseq];
  // Element offsets are 64-bit in the kernels; bound T*H*D so byte sizes fit comfortably.
  // Within one staged tile the kernels address rows with 32-bit byte offsets, which needs
  // 64 rows of stride H*D to stay far below 2^32 bytes.
  const int64_t elems = T * static_cast<int64_t>(heads) * head_dim;
  if (static_cast<int64_t>(heads) * head_dim > (int64_t(1) << 22) || elems > (int64_t(1) << 40))
    return set_error(T2V_ERR_INVALID_ARG, "heads * head_dim or T * heads * head_dim is too large");
  *total_tokens = T;
  return T2V_OK;
}

int validate_shape_qk(const int32_t* cu_q, const int32_t* cu_k, int nseq, int heads, int head_dim, float scale,
                      int64_t* tq, int64_t* tk) {
  if (int st = validate_shape(cu_q, nseq, heads, head_dim, scale, tq)) return st;
  if (cu_k == nullptr) return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens_k is NULL");
  if (int st = validate_shape(cu_k, nseq, heads, head_dim, scale, tk)) {
    return set_error(st, std::string("cu_seqlens_k: ") + last_error());
  }
  for (int s = 0; s < nseq; ++s) {
    const bool has_q = cu_q[s + 1] > cu_q[s], has_k = cu_k[s + 1] > cu_k[s];
    if (has_q != has_k)
      return set_error(T2V_ERR_INVALID_ARG, "sequence " + std::to_string(s) + (has_q ? " has queries but no keys"
                                                                                      : " has keys but no queries"));
  }
  return T2V_OK;
}

int validate_pointers(const std::vector<Range>& inputs, const std::vector<Range>& outputs) {
  auto check = [](const Range& r) -> int {
    if (r.ptr == nullptr) return set_error(T2V_ERR_INVALID_ARG, std::string(r.name) + " is NULL");
    if (reinterpret_cast<uintptr_t>(r.ptr) % 16 != 0)
      return set_error(T2V_ERR_INVALID_ARG, std::string(r.name) + " is not 16-byte aligned");
    return T2V_OK;
  };
  for (const auto& r : inputs)
    if (int st = check(r)) return st;
  for (const auto& r : outputs)
    if (int st = check(r)) return st;
  auto overlap = [](const Range& a, const Range& b) {
    const auto a0 = reinterpret_cast<uintptr_t>(a.ptr), b0 = reinterpret_cast<uintptr_t>(b.ptr);
    return a0 < b0 + static_cast<uintptr_t>(b.bytes) && b0 < a0 + static_cast<uintptr_t>(a.bytes);
  };
  for (size_t i = 0; i < outputs.size(); ++i) {
    for (const auto& in : inputs)
      if (overlap(outputs[i], in))
        return set_error(T2V_ERR_INVALID_ARG, std::string(outputs[i].name) + " overlaps input " + in.name);
    for (size_t j = i + 1; j < outputs.size(); ++j)
      if (overlap(outputs[i], outputs[j]))
        return set_error(T2V_ERR_INVALID_ARG,
                         std::string(outputs[i].name) + " overlaps output " + outputs[j].name);
  }
  return T2V_OK;
}

namespace {

// The tiles of one (sequence, head), or of one piece of its loop when the loop is split.
struct Group {
  int seq, head;
  int32_t row0, len;    // owned segment
  int32_t lrow0, llen;  // looped-over segment (or piece)
  int tiles;
  int32_t slot0 = -1;   // first partial slot of the (sequence, head); -1: not split
  int piece = 0, pieces = 1;
};

std::vector<Group> make_groups(const int32_t* cu, const int32_t* cul, int nseq, int heads, int block, int chunk) {
  std::vector<Group> g;
  int64_t next_slot = 0;
  for (int s = 0; s < nseq; ++s) {
    const int32_t L = cu[s + 1] - cu[s];
    const int32_t LL = cul[s + 1] - cul[s];
    if (L <= 0 || LL <= 0) continue;
    const int tiles = (L + block - 1) / block;
    int n = 1, step = LL;
    loop_pieces(LL, chunk, &n, &step);
    for (int h = 0; h < heads; ++h) {
      if (n == 1) {
        g.push_back({s, h, cu[s], L, cul[s], LL, tiles});
        continue;
      }
      const auto slot0 = static_cast<int32_t>(next_slot);
      next_slot += static_cast<int64_t>(tiles) * n;
      for (int j = 0; j < n; ++j)
        g.push_back({s, h, cu[s], L, cul[s] + j * step, std::min(step, LL - j * step), tiles, slot0, j, n});
    }
  }
  return g;
}

void append_tiles(std::vector<Item>& out, const Group& g, int t_begin, int t_end, int block) {
  for (int t = t_begin; t < t_end; ++t) {
    const int32_t slot = g.pieces > 1 ? g.slot0 + t * g.pieces + g.piece : -1;
    out.push_back({g.row0, g.len, t * block, g.head, g.lrow0, g.llen, slot, g.pieces});
  }
}

}  // namespace

void loop_pieces(int LL, int chunk, int* n, int* step) {
  *n = 1;
  *step = LL;
  if (chunk <= 0 || LL <= chunk) return;
  const int n0 = (LL + chunk - 1) / chunk;
  const int s = ((LL + n0 - 1) / n0 + 63) / 64 * 64;
  const int n1 = (LL + s - 1) / s;
  if (n1 <= 1) return;
  *n = n1;
  *step = s;
}

LoopSplit choose_loop_split(const int32_t* cu, const int32_t* cul, int nseq, int heads, int block, int parallel,
                            int64_t max_slots) {
  double total = 0.0, largest = 0.0;
  int32_t longest = 0;
  for (int s = 0; s < nseq; ++s) {
    const int32_t L = cu[s + 1] - cu[s], LL = cul[s + 1] - cul[s];
    if (L <= 0 || LL <= 0) continue;
    total += static_cast<double>(heads) * L * LL;
    largest = std::max(largest, static_cast<double>(std::min(block, L)) * LL);
    longest = std::max(longest, LL);
  }
  if (parallel < 1 || block < 1 || largest <= total / parallel) return {};
  const double share = std::ceil(total / (2.0 * parallel * block));
  int64_t chunk = std::max<int64_t>(kMinChunk, (static_cast<int64_t>(share) + 63) / 64 * 64);
  for (; chunk < longest; chunk *= 2) {  // widen the pieces until their partial slots fit
    int64_t slots = 0;
    for (int s = 0; s < nseq; ++s) {
      const int32_t L = cu[s + 1] - cu[s], LL = cul[s + 1] - cul[s];
      if (L <= 0 || LL <= 0) continue;
      int n = 1, step = LL;
      loop_pieces(LL, static_cast<int>(chunk), &n, &step);
      if (n > 1) slots += static_cast<int64_t>(heads) * ((L + block - 1) / block) * n;
    }
    if (slots == 0) return {};
    if (slots <= max_slots && slots <= INT32_MAX) return {static_cast<int>(chunk), slots};
  }
  return {};
}

int choose_tile_rows(const int32_t* cu, const int32_t* cul, int nseq, int heads, int wide, int narrow,
                     bool narrow_always, double narrow_max_loop, double narrow_penalty, int order, int slots,
                     std::vector<Item>* chosen) {
  if (narrow_always) return narrow;
  double work = 0.0, weighted = 0.0;
  for (int s = 0; s < nseq; ++s) {
    const double L = cu[s + 1] - cu[s], LL = cul[s + 1] - cul[s];
    if (L <= 0 || LL <= 0) continue;
    work += L * LL;
    weighted += L * LL * LL;
  }
  if (work <= 0.0 || weighted <= narrow_max_loop * work) return narrow;
  if (slots < 1) return wide;
  double ms_wide = 0.0, ms_narrow = 0.0, lb = 0.0;
  std::vector<Item> w = build_worklist(cu, cul, nseq, heads, wide, order);
  plan_makespan(w.data(), static_cast<int>(w.size()), wide, slots, &ms_wide, &lb);
  std::vector<Item> n = build_worklist(cu, cul, nseq, heads, narrow, order);
  plan_makespan(n.data(), static_cast<int>(n.size()), narrow, slots, &ms_narrow, &lb);
  const bool take_narrow = ms_narrow * narrow_penalty < ms_wide;
  if (chosen != nullptr) *chosen = std::move(take_narrow ? n : w);
  return take_narrow ? narrow : wide;
}

std::vector<Item> build_reduce_list(const int32_t* cu, const int32_t* cul, int nseq, int heads, int block,
                                    int chunk) {
  std::vector<Item> out;
  for (const Group& g : make_groups(cu, cul, nseq, heads, block, chunk))
    if (g.pieces > 1 && g.piece == 0)
      for (int t = 0; t < g.tiles; ++t)
        out.push_back({g.row0, g.len, t * block, g.head, 0, 0, g.slot0 + t * g.pieces, g.pieces});
  return out;
}

std::string check_work_items(const Item* items, int n, const int32_t* cu_own, const int32_t* cu_loop, int nseq,
                             int heads, int block, int64_t max_slots, bool reduce) {
  for (int i = 0; i < n; ++i) {
    const Item& it = items[i];
    auto bad = [&](const char* what) {
      return "item " + std::to_string(i) + " {row0 " + std::to_string(it.row0) + ", len " + std::to_string(it.len) +
             ", tile0 " + std::to_string(it.tile0) + ", head " + std::to_string(it.head) + ", lrow0 " +
             std::to_string(it.lrow0) + ", llen " + std::to_string(it.llen) + ", slot " + std::to_string(it.slot) +
             ", pieces " + std::to_string(it.pieces) + "}: " + what;
    };
    // The segment starting at row0: the last s with cu_own[s] <= row0 (empty clips before a
    // non-empty one share its start, so this is the non-empty one when there is one).
    const int s = static_cast<int>(std::upper_bound(cu_own, cu_own + nseq + 1, it.row0) - cu_own) - 1;
    if (s < 0 || s >= nseq || cu_own[s] != it.row0) return bad("row0 is not the start of a clip");
    if (it.len < 1 || it.len != cu_own[s + 1] - cu_own[s]) return bad("len is not its clip's length");
    if (it.tile0 < 0 || it.tile0 >= it.len || it.tile0 % block != 0) return bad("tile0 is outside the clip");
    if (it.head < 0 || it.head >= heads) return bad("head is out of range");
    if (reduce) {
      if (it.slot < 0 || it.pieces < 2 || static_cast<int64_t>(it.slot) + it.pieces > max_slots)
        return bad("partial slots are out of range");
      continue;
    }
    const int32_t a = cu_loop[s], b = cu_loop[s + 1];
    if (it.llen < 1 || it.lrow0 < a || static_cast<int64_t>(it.lrow0) + it.llen > b)
      return bad("looped-over rows leave the clip's segment");
    if (it.slot < 0) {
      if (it.slot != -1 || it.pieces != 1 || it.lrow0 != a || it.llen != b - a)
        return bad("an unsplit item must loop over its whole segment");
    } else if (it.pieces < 2 || it.slot >= max_slots) {
      return bad("partial slot is out of range");
    }
  }
  return std::string();
}

std::vector<Item> build_worklist(const int32_t* cu, const int32_t* cu_loop, int nseq, int heads, int block,
                                 int order, int chunk) {
  std::vector<Group> groups = make_groups(cu, cu_loop, nseq, heads, block, chunk);
  std::vector<Item> items;
  size_t n = 0;
  for (const auto& g : groups) n += g.tiles;
  items.reserve(n);
  if (order == T2V_ORDER_NATURAL) {
    for (const auto& g : groups) append_tiles(items, g, 0, g.tiles, block);
    return items;
  }
  // Longest tiles first (a tile costs its rows times the looped-over length; for
  // self-attention this is the longest clip first); ties keep pack order, so one
  // (sequence, head)'s tiles stay adjacent.
  std::stable_sort(groups.begin(), groups.end(), [](const Group& a, const Group& b) { return a.llen > b.llen; });
  // Workgroup b runs on XCD b % 8, and each XCD starts its share in increasing b, so every
  // XCD takes the same number of items. Deal whole (clip, head) groups to the least-loaded
  // XCD that has room for them and stays within an even share of the total cost, so the
  // concurrently running tiles on one XCD read the same K/V through that XCD's L2. A group
  // that fits nowhere (too many items, or too costly: few heavy groups, e.g. one long clip
  // at a few heads) is split, filling the least-loaded XCD up to its share first.
  std::vector<size_t> cap(kNumXcd);
  for (int x = 0; x < kNumXcd; ++x) cap[x] = n / kNumXcd + (static_cast<size_t>(x) < n % kNumXcd ? 1 : 0);
  std::vector<std::vector<Item>> q(kNumXcd);
  std::vector<double> load(kNumXcd, 0.0);
  double total = 0.0;
  for (const auto& g : groups) total += static_cast<double>(g.tiles) * block * g.llen;
  const double share = total / kNumXcd * (1.0 + 1e-9);
  for (const auto& g : groups) {
    const double item_cost = static_cast<double>(block) * g.llen;
    int t = 0;
    while (t < g.tiles) {
      const size_t want = static_cast<size_t>(g.tiles - t);
      int best = -1;
      for (int x = 0; x < kNumXcd; ++x)  // least-loaded XCD with room for the rest of the group
        if (cap[x] - q[x].size() >= want && load[x] + static_cast<double>(want) * item_cost <= share &&
            (best < 0 || load[x] < load[best]))
          best = x;
      size_t take = want;
      if (best < 0) {  // split: the least-loaded XCD with any room, up to its share
        for (int x = 0; x < kNumXcd; ++x)
          if (cap[x] > q[x].size() && (best < 0 || load[x] < load[best])) best = x;
        const double fit = std::floor((share - load[best]) / item_cost);
        const size_t under = fit >= 1.0 ? static_cast<size_t>(std::min(fit, 1e15)) : 1;
        take = std::min({want, cap[best] - q[best].size(), under});
      }
      append_tiles(q[best], g, t, t + static_cast<int>(take), block);
      load[best] += static_cast<double>(take) * item_cost;
      t += static_cast<int>(take);
    }
  }
  // With few groups the item-count capacity can still leave the XCDs' costs uneven. Then
  // deal single items instead (longest first, each to the least-loaded XCD with room),
  // which balances cost at the price of spreading each group's K/V over all XCDs' L2s
  // (measured: 0.6% slower where group dealing balances, 3-5% faster where it does not).
  auto imbalance = [](const std::vector<double>& l) {
    double mx = 0.0, sum = 0.0;
    for (double x : l) {
      mx = std::max(mx, x);
      sum += x;
    }
    return sum > 0.0 ? mx * static_cast<double>(l.size()) / sum : 1.0;
  };
  const double grouped = imbalance(load);
  if (grouped > 1.01) {
    std::vector<std::vector<Item>> qi(kNumXcd);
    std::vector<double> li(kNumXcd, 0.0);
    for (const auto& g : groups) {
      std::vector<Item> tiles;
      append_tiles(tiles, g, 0, g.tiles, block);
      for (const Item& it : tiles) {
        int best = -1;
        for (int x = 0; x < kNumXcd; ++x)
          if (cap[x] > qi[x].size() && (best < 0 || li[x] < li[best])) best = x;
        qi[best].push_back(it);
        li[best] += static_cast<double>(block) * it.llen;
      }
    }
    if (imbalance(li) < grouped) q.swap(qi);
  }
  items.resize(n);
  for (size_t b = 0; b < n; ++b) items[b] = q[b % kNumXcd][b / kNumXcd];
  return items;
}

RangeAllocator::RangeAllocator(uint64_t size) : size_(size / kAlign * kAlign), free_total_(size_) {
  if (size_ > 0) free_.push_back({0, size_});
}

int64_t RangeAllocator::alloc(uint64_t bytes) {
  const uint64_t need = rounded(bytes == 0 ? 1 : bytes);
  for (size_t i = 0; i < free_.size(); ++i) {
    if (free_[i].second < need) continue;
    const uint64_t off = free_[i].first;
    free_[i].first += need;
    free_[i].second -= need;
    if (free_[i].second == 0) free_.erase(free_.begin() + static_cast<std::ptrdiff_t>(i));
    free_total_ -= need;
    return static_cast<int64_t>(off);
  }
  return -1;
}

bool RangeAllocator::release(uint64_t off, uint64_t bytes) {
  const uint64_t len = rounded(bytes == 0 ? 1 : bytes);
  if (off % kAlign != 0 || off > size_ || len > size_ - off) return false;
  // First free range at or after off; the released range must fit between it and the one before.
  auto it = std::lower_bound(free_.begin(), free_.end(), std::make_pair(off, uint64_t(0)));
  if (it != free_.end() && it->first < off + len) return false;                         // overlaps a free range
  if (it != free_.begin() && std::prev(it)->first + std::prev(it)->second > off) return false;
  it = free_.insert(it, {off, len});
  free_total_ += len;
  auto next = std::next(it);
  if (next != free_.end() && it->first + it->second == next->first) {  // merge with the next range
    it->second += next->second;
    it = std::prev(free_.erase(next));
  }
  if (it != free_.begin()) {  // merge with the previous range
    auto prev = std::prev(it);
    if (prev->first + prev->second == it->first) {
      prev->second += it->second;
      free_.erase(it);
    }
  }
  return true;
}

void plan_makespan(const Item* items, int n, int block, int slots, double* makespan, double* lower_bound) {
  double total = 0.0, largest = 0.0;
  auto cost = [block](const Item& it) {
    const int rows = std::min(block, it.len - it.tile0);
    return static_cast<double>(rows) * it.llen;
  };
  for (int i = 0; i < n; ++i) {
    total += cost(items[i]);
    largest = std::max(largest, cost(items[i]));
  }
  *lower_bound = slots > 0 ? std::max(total / slots, largest) : 0.0;
  double span = 0.0;
  const int groups = (slots % kNumXcd == 0 && slots >= kNumXcd) ? kNumXcd : 1;
  const int per = slots / groups;
  for (int x = 0; x < groups && per > 0; ++x) {
    std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
    for (int s = 0; s < per; ++s) free_at.push(0.0);
    for (int i = x; i < n; i += groups) {
      const double t0 = free_at.top();
      free_at.pop();
      free_at.push(t0 + cost(items[i]));
    }
    while (free_at.size() > 1) free_at.pop();
    span = std::max(span, free_at.top());
  }
  *makespan = span;
}

}  // namespace t2v

extern "C" {

const char* t2v_last_error(void) { return t2v::last_error(); }

const char* t2v_version(void) { return "libt2vattn 0.1 (gfx950)"; }

int t2v_build_worklist(const int32_t* cu_seqlens, int nseq, int heads, int block, int order,
                       int32_t* items_out, int capacity, int* n_items_out) {
  if (n_items_out == nullptr) return t2v::set_error(T2V_ERR_INVALID_ARG, "n_items_out is NULL");
  *n_items_out = 0;
  if (nseq < 0 || cu_seqlens == nullptr || heads < 1 || block < 1)
    return t2v::set_error(T2V_ERR_INVALID_ARG, "bad nseq, cu_seqlens, heads or block");
  if (order != T2V_ORDER_NATURAL && order != T2V_ORDER_LONGEST_FIRST)
    return t2v::set_error(T2V_ERR_INVALID_ARG, "unknown order");
  if (cu_seqlens[0] != 0) return t2v::set_error(T2V_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  for (int s = 0; s < nseq; ++s)
    if (cu_seqlens[s + 1] < cu_seqlens[s])
      return t2v::set_error(T2V_ERR_INVALID_ARG, "cu_seqlens must be non-decreasing");
  std::vector<t2v::Item> items = t2v::build_worklist(cu_seqlens, cu_seqlens, nseq, heads, block, order);
  if (items.size() > static_cast<size_t>(INT32_MAX))
    return t2v::set_error(T2V_ERR_INVALID_ARG, "too many work items");
  *n_items_out = static_cast<int>(items.size());
  if (items_out == nullptr) return T2V_OK;
  if (capacity < static_cast<int>(items.size()))
    return t2v::set_error(T2V_ERR_INVALID_ARG, "capacity too small");
  for (size_t i = 0; i < items.size(); ++i) {  // self-attention: (row0, len, tile0, head) per item
    items_out[4 * i + 0] = items[i].row0;
    items_out[4 * i + 1] = items[i].len;
    items_out[4 * i + 2] = items[i].tile0;
    items_out[4 * i + 3] = items[i].head;
  }
  return T2V_OK;
}

int t2v_plan_makespan(const int32_t* items, int n_items, int block, int slots, double* makespan_out,
                      double* lower_bound_out) {
  if ((items == nullptr && n_items > 0) || n_items < 0 || block < 1 || slots < 1 || makespan_out == nullptr ||
      lower_bound_out == nullptr)
    return t2v::set_error(T2V_ERR_INVALID_ARG, "bad plan arguments");
  std::vector<t2v::Item> it(static_cast<size_t>(n_items));
  for (int i = 0; i < n_items; ++i) {  // self-attention items: the loop segment is the clip
    const int32_t* r = items + 4 * static_cast<size_t>(i);
    it[i] = {r[0], r[1], r[2], r[3], r[0], r[1], -1, 1};
  }
  t2v::plan_makespan(it.data(), n_items, block, slots, makespan_out, lower_bound_out);
  return T2V_OK;
}

}  // extern "C"
