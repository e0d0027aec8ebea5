// Randomised exercise of the host-side code of libt2vattn (tile scheduler and its loop
// split, makespan model, argument validation, cascade planner, work-list pool allocator, the
// checked library's work-list checks), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py. Every check that fails prints
// a line; the exit status is the number of failed checks (sanitizer reports abort earlier).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <random>
#include <string>
#include <vector>

#include "../include/t2vattn.h"
#include "../paper_2607_01701_amd/csrc/t2v_host.h"

static int g_failed = 0;
#define CHECK(cond, what)                                              \
  do {                                                                 \
    if (!(cond)) {                                                     \
      ++g_failed;                                                      \
      std::printf("FAIL %s:%d %s\n", __FILE__, __LINE__, (what));      \
    }                                                                  \
  } while (0)

static std::vector<int32_t> random_cu(std::mt19937& rng, int nseq, int max_len) {
  std::vector<int32_t> cu(nseq + 1, 0);
  std::uniform_int_distribution<int> len(0, max_len), zero(0, 4);
  for (int s = 0; s < nseq; ++s) cu[s + 1] = cu[s] + (zero(rng) == 0 ? 0 : len(rng));
  return cu;
}

// Work lists: every (clip, head, tile) exactly once, tiles cover the clip, a short buffer
// is refused, and the makespan model respects its own lower bound.
static void worklists(std::mt19937& rng) {
  for (int rep = 0; rep < 300; ++rep) {
    const int nseq = std::uniform_int_distribution<int>(0, 40)(rng);
    const int heads = std::uniform_int_distribution<int>(1, 8)(rng);
    const int block = rep % 2 ? 128 : 256;
    const int order = rep % 3 == 0 ? T2V_ORDER_NATURAL : T2V_ORDER_LONGEST_FIRST;
    const std::vector<int32_t> cu = random_cu(rng, nseq, 5000);
    int n = -1;
    CHECK(t2v_build_worklist(cu.data(), nseq, heads, block, order, nullptr, 0, &n) == T2V_OK, "count query");
    int64_t expect = 0;
    for (int s = 0; s < nseq; ++s) expect += int64_t(heads) * ((cu[s + 1] - cu[s] + block - 1) / block);
    CHECK(n == expect, "item count");
    std::vector<int32_t> items(4 * static_cast<size_t>(n) + 4, -7);
    if (n > 0) {
      int m = 0;
      CHECK(t2v_build_worklist(cu.data(), nseq, heads, block, order, items.data(), n - 1, &m) ==
                T2V_ERR_INVALID_ARG, "short buffer refused");
    }
    CHECK(t2v_build_worklist(cu.data(), nseq, heads, block, order, items.data(), n, &n) == T2V_OK, "fill");
    CHECK(items[4 * static_cast<size_t>(n)] == -7, "no write past the items");
    std::vector<std::vector<int>> seen(static_cast<size_t>(nseq) * heads);
    for (int i = 0; i < n; ++i) {
      const int32_t* r = &items[4 * static_cast<size_t>(i)];
      int s = -1;
      for (int j = 0; j < nseq; ++j)
        if (cu[j] == r[0] && cu[j + 1] - cu[j] == r[1]) s = j;
      CHECK(s >= 0 && r[3] >= 0 && r[3] < heads && r[2] >= 0 && r[2] < r[1] && r[2] % block == 0, "item fields");
      if (s >= 0 && r[3] >= 0 && r[3] < heads) seen[static_cast<size_t>(s) * heads + r[3]].push_back(r[2]);
    }
    for (int s = 0; s < nseq; ++s)
      for (int h = 0; h < heads; ++h) {
        std::vector<int>& t = seen[static_cast<size_t>(s) * heads + h];
        const int L = cu[s + 1] - cu[s];
        std::vector<int> want;
        for (int r0 = 0; r0 < L; r0 += block) want.push_back(r0);
        std::sort(t.begin(), t.end());
        CHECK(t == want, "tiles of a (clip, head) are each present once");
      }
    for (int slots : {1, 7, 256}) {
      double ms = -1.0, lb = -1.0;
      CHECK(t2v_plan_makespan(items.data(), n, block, slots, &ms, &lb) == T2V_OK, "makespan");
      CHECK(ms >= lb - 1e-9 * (1.0 + lb) && lb >= 0.0, "makespan >= lower bound");
    }
  }
}

// Loop split: every (sequence, head, tile) loop is covered once by its pieces, pieces are
// 64-row multiples but the last, partial slots are unique and consecutive per split tile
// as its reduce item says, and the chosen split respects its slot cap.
static void loop_split(std::mt19937& rng) {
  int chosen = 0;
  for (int rep = 0; rep < 400; ++rep) {
    const int LL = std::uniform_int_distribution<int>(1, 50000)(rng);
    const int chunk = std::uniform_int_distribution<int>(-1, 9000)(rng);
    int n = 0, step = 0;
    t2v::loop_pieces(LL, chunk, &n, &step);
    const bool none = chunk <= 0 || LL <= chunk;
    CHECK(n >= 1 && (n == 1) == (step == LL), "pieces");
    CHECK(!none || n == 1, "no split at or below the chunk");
    CHECK(n == 1 || (step % 64 == 0 && static_cast<int64_t>(n - 1) * step < LL &&
                     static_cast<int64_t>(n) * step >= LL), "pieces cover the loop");
  }
  for (int rep = 0; rep < 200; ++rep) {
    const int nseq = std::uniform_int_distribution<int>(1, 12)(rng);
    const int heads = std::uniform_int_distribution<int>(1, 4)(rng);
    const int block = 128;
    const std::vector<int32_t> own = random_cu(rng, nseq, 400), loop0 = random_cu(rng, nseq, 30000);
    std::vector<int32_t> loop(loop0);  // sequences with keys but no queries get one query
    for (int s = 0, add = 0; s < nseq; ++s) {
      if (own[s + 1] > own[s] && loop0[s + 1] == loop0[s]) ++add;
      loop[s + 1] = loop0[s + 1] + add;
    }
    const int parallel = rep % 3 == 0 ? 1 : 256;
    const int64_t cap = rep % 4 == 0 ? 7 : 1 << 20;
    const t2v::LoopSplit sp = t2v::choose_loop_split(own.data(), loop.data(), nseq, heads, block, parallel, cap);
    CHECK(sp.chunk == 0 || (sp.chunk >= t2v::kMinChunk && sp.slots >= 2 && sp.slots <= cap), "split choice");
    CHECK(parallel > 1 || sp.chunk == 0, "one worker: no split");
    chosen += sp.chunk > 0 ? 1 : 0;
    const int chunk = sp.chunk > 0 ? sp.chunk : (rep % 2 ? 2048 : 0);
    const std::vector<t2v::Item> items =
        t2v::build_worklist(own.data(), loop.data(), nseq, heads, block, T2V_ORDER_LONGEST_FIRST, chunk);
    const std::vector<t2v::Item> red = t2v::build_reduce_list(own.data(), loop.data(), nseq, heads, block, chunk);
    int64_t slots = 0;
    for (const auto& r : red) slots += r.pieces;
    if (sp.chunk > 0) CHECK(slots == sp.slots, "slot count matches the choice");
    std::vector<int> slot_seen(static_cast<size_t>(slots), 0);
    for (const auto& it : items) {
      CHECK(it.llen >= 1, "piece has rows");
      if (it.slot >= 0) {
        CHECK(it.slot < slots && it.pieces >= 2, "slot in range");
        if (it.slot < slots) ++slot_seen[static_cast<size_t>(it.slot)];
      } else {
        CHECK(it.pieces == 1, "unsplit item");
      }
    }
    for (int v : slot_seen) CHECK(v == 1, "every slot written by one item");
    for (int s = 0; s < nseq; ++s) {
      const int L = own[s + 1] - own[s], LL = loop[s + 1] - loop[s];
      if (L <= 0 || LL <= 0) continue;
      for (int h = 0; h < heads; ++h)
        for (int t0 = 0; t0 < L; t0 += block) {
          std::vector<std::pair<int, int>> ranges;
          std::vector<int32_t> tslots;
          for (const auto& it : items)
            if (it.row0 == own[s] && it.len == L && it.head == h && it.tile0 == t0) {
              ranges.push_back({it.lrow0, it.llen});
              tslots.push_back(it.slot);
            }
          std::sort(ranges.begin(), ranges.end());
          std::sort(tslots.begin(), tslots.end());
          int64_t at = loop[s];
          for (const auto& r : ranges) {
            CHECK(r.first == at, "pieces are contiguous");
            at = static_cast<int64_t>(r.first) + r.second;
          }
          CHECK(at == loop[s + 1], "pieces end at the loop end");
          int nr = 0;
          for (const auto& r : red)
            if (r.row0 == own[s] && r.head == h && r.tile0 == t0) {
              ++nr;
              CHECK(r.pieces == static_cast<int>(ranges.size()) && tslots.front() == r.slot &&
                        tslots.back() == r.slot + r.pieces - 1, "reduce item names the tile's slots");
            }
          CHECK(nr == (ranges.size() > 1 ? 1 : 0), "one reduce item per split tile");
        }
    }
  }
  std::printf("loop split chosen in %d of 200 packs\n", chosen);
  CHECK(chosen >= 20, "the random packs exercise the split");
}

// Tile choice: narrow when forced by head_dim or short loops; on long loops, narrow only
// where the wide list leaves the last round part-empty.
static void tile_choice() {
  const std::vector<int32_t> short_cu = {0, 300, 600};
  CHECK(t2v::choose_tile_rows(short_cu.data(), short_cu.data(), 2, 24, 256, 128, false, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 256) == 128, "short loops: narrow");
  const std::vector<int32_t> one = {0, 75600};
  CHECK(t2v::choose_tile_rows(one.data(), one.data(), 1, 24, 256, 128, true, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 256) == 128, "narrow_always");
  CHECK(t2v::choose_tile_rows(one.data(), one.data(), 1, 24, 256, 128, false, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 256) == 256, "long clip, 24 heads: wide");
  CHECK(t2v::choose_tile_rows(one.data(), one.data(), 1, 3, 256, 128, false, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 256) == 128, "long clip, 3 heads: narrow (888 wide tiles)");
  CHECK(t2v::choose_tile_rows(one.data(), one.data(), 1, 3, 256, 128, false, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 0) == 256, "no slots known: wide");
  const std::vector<int32_t> none = {0, 0};
  CHECK(t2v::choose_tile_rows(none.data(), none.data(), 1, 3, 256, 128, false, 1536.0, 1.04,
                              T2V_ORDER_LONGEST_FIRST, 256) == 128, "empty pack");
}

// Validation: each rejected input yields the error it should, never a crash.
static void validation(std::mt19937& rng) {
  int64_t T = 0, Tk = 0;
  const std::vector<int32_t> good = {0, 5, 5, 12};
  CHECK(t2v::validate_shape(good.data(), 3, 2, 128, 0.1f, &T) == T2V_OK && T == 12, "valid shape");
  const std::vector<int32_t> dec = {0, 5, 4};
  CHECK(t2v::validate_shape(dec.data(), 2, 2, 128, 0.1f, &T) == T2V_ERR_INVALID_ARG, "decreasing offsets");
  CHECK(t2v::validate_shape(good.data(), 3, 0, 128, 0.1f, &T) == T2V_ERR_INVALID_ARG, "no heads");
  CHECK(t2v::validate_shape(good.data(), 3, 2, 96, 0.1f, &T) == T2V_ERR_UNSUPPORTED, "head_dim");
  CHECK(t2v::validate_shape(good.data(), 3, 2, 128, INFINITY, &T) == T2V_ERR_INVALID_ARG, "scale");
  CHECK(t2v::validate_shape(nullptr, 3, 2, 128, 0.1f, &T) == T2V_ERR_INVALID_ARG, "null offsets");
  const std::vector<int32_t> keys = {0, 3, 4, 9};  // sequence 1: a key but no queries
  CHECK(t2v::validate_shape_qk(good.data(), keys.data(), 3, 2, 64, 0.1f, &T, &Tk) == T2V_ERR_INVALID_ARG,
        "keys without queries");
  alignas(64) static char buf[4096];
  std::vector<t2v::Range> in = {{buf, 1024, "a"}}, out = {{buf + 512, 1024, "b"}};
  CHECK(t2v::validate_pointers(in, out) == T2V_ERR_INVALID_ARG, "overlap");
  out = {{buf + 1024, 1024, "b"}};
  CHECK(t2v::validate_pointers(in, out) == T2V_OK, "disjoint");
  out = {{buf + 1028, 16, "b"}};
  CHECK(t2v::validate_pointers(in, out) == T2V_ERR_INVALID_ARG, "misaligned");
  for (int rep = 0; rep < 200; ++rep) {  // random offsets, some of them invalid
    const int nseq = std::uniform_int_distribution<int>(0, 30)(rng);
    std::vector<int32_t> cu = random_cu(rng, nseq, 300);
    if (nseq > 0 && rep % 4 == 0) cu[1 + rng() % nseq] -= 1000;
    const int st = t2v::validate_shape(cu.data(), nseq, 1 + rng() % 4, rep % 2 ? 64 : 128, 0.2f, &T);
    CHECK(st == T2V_OK || st == T2V_ERR_INVALID_ARG, "validation status");
  }
}

// Planner: schedules respect precedence and the GPU count; a cycle is refused.
static void planner(std::mt19937& rng) {
  const std::vector<int32_t> K = {1, 2, 4, 8};
  for (int rep = 0; rep < 60; ++rep) {
    const int n = std::uniform_int_distribution<int>(1, 30)(rng);
    const int N = std::uniform_int_distribution<int>(1, 16)(rng);
    std::vector<int32_t> ptr(n + 1, 0), idx;
    for (int c = 0; c < n; ++c) {
      for (int p = 0; p < c; ++p)
        if (rng() % 5 == 0) idx.push_back(p);
      ptr[c + 1] = static_cast<int32_t>(idx.size());
    }
    if (idx.empty()) idx.push_back(0);
    std::vector<double> lat(static_cast<size_t>(n) * K.size()), mem(lat.size());
    std::uniform_real_distribution<double> u(0.1, 2.0);
    for (int c = 0; c < n; ++c)
      for (size_t j = 0; j < K.size(); ++j) {
        lat[c * K.size() + j] = u(rng) / K[j] + 0.05 * K[j];
        mem[c * K.size() + j] = u(rng) / K[j];
      }
    std::vector<int32_t> deg(n, 0);
    std::vector<double> start(n, -1.0);
    double T = -1.0;
    const int st = t2v_plan_cascades(n, ptr.data(), idx.data(), static_cast<int>(K.size()), K.data(), lat.data(),
                                     mem.data(), 2.0, N, 16, 20, 0.05, 2, 1234u + rep, deg.data(), start.data(), &T);
    CHECK(st == T2V_OK, "plan");
    if (st != T2V_OK) continue;
    double tmax = 0.0;
    std::vector<double> end(n);
    for (int c = 0; c < n; ++c) {
      size_t j = 0;
      while (j < K.size() && K[j] != deg[c]) ++j;
      CHECK(j < K.size() && deg[c] <= N, "degree in K and <= N");
      end[c] = start[c] + lat[c * K.size() + (j < K.size() ? j : 0)];
      tmax = std::max(tmax, end[c]);
      CHECK(start[c] >= 0.0, "start >= 0");
    }
    for (int c = 0; c < n; ++c)
      for (int e = ptr[c]; e < ptr[c + 1]; ++e) CHECK(start[c] >= end[idx[e]] - 1e-9, "precedence");
    CHECK(std::fabs(tmax - T) <= 1e-9 * (1.0 + T), "makespan is the last end");
    for (int c = 0; c < n; ++c) {  // GPUs in use when cascade c starts
      int used = 0;
      for (int d = 0; d < n; ++d)
        if (start[d] <= start[c] + 1e-12 && start[c] < end[d] - 1e-12) used += deg[d];
      CHECK(used <= N, "at most N GPUs in use");
    }
  }
  const std::vector<int32_t> ptr = {0, 1, 2}, idx = {1, 0};  // 0 <- 1 and 1 <- 0
  const std::vector<int32_t> deg = {1, 1};
  const std::vector<double> lat = {1.0, 1.0};
  std::vector<double> start(2);
  double T = 0.0;
  CHECK(t2v_list_schedule(2, ptr.data(), idx.data(), deg.data(), lat.data(), 2, start.data(), &T) ==
            T2V_ERR_INVALID_ARG, "cycle refused");
}

// The work-list memory pool's range allocator against a byte-map model: every allocation
// is disjoint from every live one and inside the chunk, double or foreign releases are
// refused, the free byte count is exact, and freeing everything leaves one range.
static void range_allocator(std::mt19937& rng) {
  for (int rep = 0; rep < 40; ++rep) {
    const uint64_t size = t2v::RangeAllocator::kAlign * std::uniform_int_distribution<uint64_t>(1, 400)(rng);
    t2v::RangeAllocator a(size);
    std::vector<int> owner(size / t2v::RangeAllocator::kAlign, -1);  // allocation id per 256-byte unit
    std::vector<std::pair<uint64_t, uint64_t>> live;                 // (offset, bytes)
    for (int op = 0; op < 600; ++op) {
      if (live.empty() || std::uniform_int_distribution<int>(0, 2)(rng) > 0) {
        const uint64_t bytes = std::uniform_int_distribution<uint64_t>(0, 9000)(rng);
        const int64_t off = a.alloc(bytes);
        const uint64_t units = t2v::RangeAllocator::rounded(bytes == 0 ? 1 : bytes) / t2v::RangeAllocator::kAlign;
        if (off < 0) {  // refused: no free run of that many units (first fit scans all of them)
          uint64_t run = 0, best = 0;
          for (int o : owner) {
            run = o < 0 ? run + 1 : 0;
            best = std::max(best, run);
          }
          CHECK(best < units, "allocation refused although a free run exists");
          continue;
        }
        CHECK(static_cast<uint64_t>(off) % t2v::RangeAllocator::kAlign == 0, "aligned offset");
        const uint64_t u0 = static_cast<uint64_t>(off) / t2v::RangeAllocator::kAlign;
        CHECK(u0 + units <= owner.size(), "allocation inside the chunk");
        for (uint64_t u = u0; u < u0 + units && u < owner.size(); ++u) {
          CHECK(owner[u] < 0, "allocation disjoint from live ones");
          owner[u] = static_cast<int>(live.size());
        }
        live.push_back({static_cast<uint64_t>(off), bytes});
      } else {
        const size_t i = std::uniform_int_distribution<size_t>(0, live.size() - 1)(rng);
        const auto r = live[i];
        CHECK(a.release(r.first, r.second), "release of a live range");
        CHECK(!a.release(r.first, r.second), "double release refused");
        const uint64_t units = t2v::RangeAllocator::rounded(r.second == 0 ? 1 : r.second) / t2v::RangeAllocator::kAlign;
        for (uint64_t u = r.first / t2v::RangeAllocator::kAlign; u < r.first / t2v::RangeAllocator::kAlign + units; ++u)
          owner[u] = -1;
        live.erase(live.begin() + static_cast<std::ptrdiff_t>(i));
        for (size_t j = 0; j < live.size(); ++j) {  // renumber owners after the erase
          const uint64_t n = t2v::RangeAllocator::rounded(live[j].second == 0 ? 1 : live[j].second) /
                             t2v::RangeAllocator::kAlign;
          for (uint64_t u = live[j].first / t2v::RangeAllocator::kAlign; u < live[j].first / t2v::RangeAllocator::kAlign + n; ++u)
            owner[u] = static_cast<int>(j);
        }
      }
      uint64_t free_units = 0;
      for (int o : owner) free_units += o < 0 ? 1 : 0;
      CHECK(a.free_bytes() == free_units * t2v::RangeAllocator::kAlign, "free byte count");
    }
    CHECK(!a.release(size, 256), "release past the chunk refused");
    for (const auto& r : live) CHECK(a.release(r.first, r.second), "final release");
    CHECK(a.free_bytes() == a.size() && a.free_ranges() == (a.size() > 0 ? 1u : 0u), "everything coalesces");
  }
}

// Work-list checks of the checked library: lists the scheduler builds pass (self and cross
// offsets, with and without the loop split); one corrupted field of one item is reported.
static void work_item_checks(std::mt19937& rng) {
  int corrupted = 0;
  for (int rep = 0; rep < 150; ++rep) {
    const int nseq = std::uniform_int_distribution<int>(1, 10)(rng);
    const int heads = std::uniform_int_distribution<int>(1, 4)(rng);
    const int block = 128;
    const std::vector<int32_t> own = random_cu(rng, nseq, 700);
    std::vector<int32_t> loop = own;
    if (rep % 2) {  // cross offsets: every sequence with rows gets at least one looped-over row
      loop = random_cu(rng, nseq, 9000);
      for (int s = 0, add = 0; s < nseq; ++s) {
        if (own[s + 1] > own[s] && loop[s + 1] + add == loop[s]) ++add;
        loop[s + 1] += add;
      }
    }
    const int chunk = rep % 3 == 0 ? 2048 : 0;
    std::vector<t2v::Item> items =
        t2v::build_worklist(own.data(), loop.data(), nseq, heads, block, T2V_ORDER_LONGEST_FIRST, chunk);
    std::vector<t2v::Item> red = t2v::build_reduce_list(own.data(), loop.data(), nseq, heads, block, chunk);
    int64_t slots = 0;
    for (const auto& r : red) slots += r.pieces;
    const int n = static_cast<int>(items.size());
    CHECK(t2v::check_work_items(items.data(), n, own.data(), loop.data(), nseq, heads, block, slots, false).empty(),
          "a scheduler list passes");
    CHECK(t2v::check_work_items(red.data(), static_cast<int>(red.size()), own.data(), loop.data(), nseq, heads,
                                block, slots, true).empty(), "a reduce list passes");
    if (n == 0) continue;
    const int i = std::uniform_int_distribution<int>(0, n - 1)(rng);
    const t2v::Item good = items[i];
    const bool split = good.slot >= 0;
    int s = 0;  // the item's clip (the last with this start: earlier empty clips share it)
    for (int j = 0; j < nseq; ++j)
      if (own[j] == good.row0 && own[j + 1] > own[j]) s = j;
    const int32_t before = loop[s] - 1, past = loop[s + 1] - good.lrow0 + 1;  // one row outside the segment
    const std::vector<std::pair<const char*, t2v::Item>> bad = {
        {"row0 is not the start", {good.row0 + 1, good.len, good.tile0, good.head, good.lrow0, good.llen, good.slot,
                                   good.pieces}},
        {"len is not", {good.row0, good.len + 1, good.tile0, good.head, good.lrow0, good.llen, good.slot, good.pieces}},
        {"tile0 is outside", {good.row0, good.len, good.len + (block - good.len % block) % block, good.head,
                              good.lrow0, good.llen, good.slot, good.pieces}},
        {"tile0 is outside", {good.row0, good.len, good.tile0 + 1, good.head, good.lrow0, good.llen, good.slot,
                              good.pieces}},
        {"head is out of range", {good.row0, good.len, good.tile0, heads, good.lrow0, good.llen, good.slot,
                                  good.pieces}},
        {"head is out of range", {good.row0, good.len, good.tile0, -1, good.lrow0, good.llen, good.slot, good.pieces}},
        {"looped-over rows leave", {good.row0, good.len, good.tile0, good.head, before, good.llen, good.slot,
                                    good.pieces}},
        {"looped-over rows leave", {good.row0, good.len, good.tile0, good.head, good.lrow0, past, good.slot,
                                    good.pieces}},
        {split ? "partial slot is out of range" : "an unsplit item",
         {good.row0, good.len, good.tile0, good.head, good.lrow0, good.llen, split ? static_cast<int32_t>(slots) : -1,
          split ? good.pieces : 2}},
    };
    for (const auto& b : bad) {
      std::vector<t2v::Item> copy = items;
      copy[i] = b.second;
      const std::string why =
          t2v::check_work_items(copy.data(), n, own.data(), loop.data(), nseq, heads, block, slots, false);
      CHECK(why.find(b.first) != std::string::npos, ("corrupted item reported: " + std::string(b.first)).c_str());
      ++corrupted;
    }
    if (!red.empty()) {
      std::vector<t2v::Item> copy = red;
      copy.back().pieces += 1;  // one slot past the last
      CHECK(t2v::check_work_items(copy.data(), static_cast<int>(copy.size()), own.data(), loop.data(), nseq, heads,
                                  block, slots, true).find("partial slots") != std::string::npos,
            "reduce item past the slots reported");
    }
  }
  std::printf("work-item checks: %d corrupted lists reported\n", corrupted);
}

int main() {
  std::mt19937 rng(20260);
  work_item_checks(rng);
  range_allocator(rng);
  worklists(rng);
  loop_split(rng);
  tile_choice();
  validation(rng);
  planner(rng);
  std::printf("host sanitizer driver: %d failed checks\n", g_failed);
  return g_failed;
}
