// C ABI of libt2vattn: argument validation, the device work-list cache, and launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <list>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/t2vattn.h"
#include "t2v_host.h"
#include "t2v_kernels.h"

// The no-allocation backward's scratch (see attn_bwd_noalloc_impl): one per GPU, held until
// the process ends. Host code must not use this name as a device address.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace t2v {
namespace {

int hip_fail(hipError_t e, const char* what) {
  return set_error(T2V_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// The scheduler order: longest clip first unless T2V_ORDER=natural (for ablations).
int order_from_env() {
  const char* s = std::getenv("T2V_ORDER");
  if (s != nullptr && std::strcmp(s, "natural") == 0) return T2V_ORDER_NATURAL;
  return T2V_ORDER_LONGEST_FIRST;
}

// Forward / dQ tile shape: narrow (4 waves, 128 queries) or wide (8 waves, 256 queries).
// Narrow tiles fit two workgroups per CU at D = 128 and three at D = 64, so one workgroup's
// Q loads and output stores overlap another's MFMA work; wide tiles stage each K/V tile
// once per 256 queries. Measured on MI355X (uniform packs): at D = 64 narrow is faster at
// every length (8-19% forward, 4-12% dQ); at D = 128 the forward crosses over near 1,536
// keys and dQ near 8,192-16,384, beyond which narrow tiles cost about 4% (forward) and 1%
// (dQ) more per unit of work. choose_tile_rows compares the work-weighted key length with
// those crossovers and, above them, the list-scheduling makespans of both work lists with
// that penalty: a pack of few tiles per CU (one GPU's share of a long clip under head
// sharding) loses more to a part-empty last round of wide tiles. T2V_QTILE=wide or narrow
// forces one (ablations and tests).
struct TileRule {
  int kind = 0;  // 0: dK/dV (one tile shape), 1: forward, 2: dQ
  int wide = 0, narrow = 0;
  bool narrow_always = false;
  double max_loop = 0.0, penalty = 1.0;
  int forced = 0;  // 0: chosen by the rule, 1: wide, 2: narrow
  bool same(const TileRule& o) const {
    return kind == o.kind && wide == o.wide && narrow == o.narrow && narrow_always == o.narrow_always &&
           forced == o.forced;
  }
};

int forced_tiles() {
  const char* s = std::getenv("T2V_QTILE");
  if (s != nullptr && std::strcmp(s, "wide") == 0) return 1;
  if (s != nullptr && std::strcmp(s, "narrow") == 0) return 2;
  return 0;
}

TileRule fwd_rule(int head_dim) {
  TileRule r;
  r.kind = 1;
  r.wide = fwd_tile_rows(head_dim, false);
  r.narrow = fwd_tile_rows(head_dim, true);
  r.narrow_always = head_dim == 64;
  r.max_loop = 1536.0;
  r.penalty = 1.04;
  r.forced = forced_tiles();
  return r;
}

TileRule dq_rule(int head_dim) {
  TileRule r;
  r.kind = 2;
  r.wide = dq_tile_rows(head_dim, false);
  r.narrow = dq_tile_rows(head_dim, true);
  r.narrow_always = head_dim == 64;
  r.max_loop = 8192.0;
  r.penalty = 1.01;
  r.forced = forced_tiles();
  return r;
}

TileRule dkdv_rule(int head_dim) {
  TileRule r;
  r.wide = r.narrow = dkdv_tile_rows(head_dim);
  return r;
}

// T2V_PERSISTENT=1 launches the forward and dK/dV kernels on a persistent grid (as many
// workgroups as the GPU holds at once, each looping over the work list with a stride of the
// grid); the default is one workgroup per work item. Results are bitwise equal either way.
// (The dQ kernel always runs one workgroup per item: its looping form would spill.)
bool persistent_enabled() {
  const char* s = std::getenv("T2V_PERSISTENT");
  return s != nullptr && std::strcmp(s, "1") == 0;
}

// T2V_SPLIT=off disables the dK/dV loop split (for ablations).
bool split_enabled() {
  const char* s = std::getenv("T2V_SPLIT");
  return s == nullptr || std::strcmp(s, "off") != 0;
}

int cu_count() {
  int device = 0, n = 0;
  if (hipGetDevice(&device) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return n;
}

// T2V_LOG=1: one line on stderr per new work list (items, predicted makespan, bound).
bool log_enabled() {
  const char* s = std::getenv("T2V_LOG");
  return s != nullptr && std::strcmp(s, "1") == 0;
}

// T2V_TEST_FAIL_ALLOC=1 makes the work-list allocation fail, so callers can exercise the
// T2V_ERR_OOM path (nothing is launched and the cache is unchanged).
bool fail_alloc_for_test() {
  const char* s = std::getenv("T2V_TEST_FAIL_ALLOC");
  return s != nullptr && std::strcmp(s, "1") == 0;
}

// cu_seqlens must be host memory: the scheduler reads it on the host.
int check_host_pointer(const int32_t* cu) {
  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof(attr));
  const hipError_t e = hipPointerGetAttributes(&attr, cu);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // plain pageable host memory is not known to HIP
    return T2V_OK;
  }
  if (attr.type == hipMemoryTypeDevice)
    return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens must be a host pointer, got device memory");
  return T2V_OK;
}

// Both offset arrays are read on the host (validation, scheduling), so they are checked to
// be host memory before anything dereferences them, including the T = 0 early return.
int check_offsets_on_host(const int32_t* cu_q, const int32_t* cu_k) {
  if (cu_q == nullptr) return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (int st = check_host_pointer(cu_q)) return st;
  if (cu_k != cu_q) {
    if (cu_k == nullptr) return set_error(T2V_ERR_INVALID_ARG, "cu_seqlens_k is NULL");
    if (int st = check_host_pointer(cu_k)) return st;
  }
  return T2V_OK;
}

// Memory for work lists, per device: device chunks hold the lists the kernels read, pinned
// host chunks stage their uploads. Lists are carved out of the chunks by RangeAllocator, so a
// new list costs no hipMalloc / hipHostMalloc once the chunks are large enough (a chunk is
// added, at twice the size of the last, only when none has room). A range is handed back
// only after every event recorded behind its readers has completed: the upload's event for
// a staging range, and the last launch on each stream that read a device range. Nothing
// here waits for the device.
class ListPool {
 public:
  struct Block {
    int chunk = -1;
    uint64_t off = 0, bytes = 0;
    void* ptr = nullptr;
  };
  explicit ListPool(bool pinned) : pinned_(pinned) {}

  // Caller holds mu(). Returns T2V_OK and a block of `bytes`, or T2V_ERR_OOM.
  int alloc(uint64_t bytes, Block* out) {
    if (fail_alloc_for_test()) return set_error(T2V_ERR_OOM, "allocation of work-list memory failed (forced)");
    if (try_alloc(bytes, out)) return T2V_OK;
    reclaim();
    if (try_alloc(bytes, out)) return T2V_OK;
    uint64_t size = last_size_ == 0 ? (pinned_ ? kFirstPinned : kFirstDevice) : 2 * last_size_;
    while (size < RangeAllocator::rounded(bytes)) size *= 2;
    void* base = nullptr;
    const hipError_t e = pinned_ ? hipHostMalloc(&base, size, hipHostMallocDefault) : hipMalloc(&base, size);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return set_error(T2V_ERR_OOM, pinned_ ? "hipHostMalloc of work-list staging failed"
                                            : "hipMalloc of work-list memory failed");
    }
    chunks_.push_back({base, RangeAllocator(size)});
    last_size_ = size;
    return try_alloc(bytes, out) ? T2V_OK : set_error(T2V_ERR_OOM, "work-list pool");
  }

  // Caller holds mu(). The block returns to its chunk once `events` (taken over) complete.
  void release_after(const Block& b, std::vector<hipEvent_t> events) {
    if (b.chunk < 0) {
      recycle_events(events);
      return;
    }
    pending_.push_back({b, std::move(events)});
  }

  // Caller holds mu(). An event from the pool (or a new one), for recording.
  hipError_t take_event(hipEvent_t* ev) {
    if (!events_.empty()) {
      *ev = events_.back();
      events_.pop_back();
      return hipSuccess;
    }
    return hipEventCreateWithFlags(ev, hipEventDisableTiming);
  }
  void recycle_events(std::vector<hipEvent_t>& evs) {
    for (hipEvent_t e : evs) events_.push_back(e);
    evs.clear();
  }

  // Caller holds the lock and has synchronised the device: returns every pending block and
  // frees each chunk that no live block uses (a list still held by a call in progress keeps
  // its chunk), and the idle events.
  void trim_after_sync() {
    reclaim();
    for (auto& c : chunks_) {
      if (c.base == nullptr || c.alloc.free_bytes() != c.alloc.size()) continue;
      if (pinned_)
        (void)hipHostFree(c.base);
      else
        (void)hipFree(c.base);
      c.base = nullptr;
      c.alloc = RangeAllocator(0);  // an empty slot: indices of live blocks stay valid
    }
    for (hipEvent_t e : events_) (void)hipEventDestroy(e);
    events_.clear();
  }

 private:
  static constexpr uint64_t kFirstDevice = 4u << 20, kFirstPinned = 2u << 20;
  struct Chunk {
    void* base;
    RangeAllocator alloc;
  };
  struct Pending {
    Block block;
    std::vector<hipEvent_t> events;
  };
  bool try_alloc(uint64_t bytes, Block* out) {
    for (int c = static_cast<int>(chunks_.size()) - 1; c >= 0; --c) {  // newest (largest) chunk first
      const int64_t off = chunks_[c].alloc.alloc(bytes);
      if (off < 0) continue;
      *out = {c, static_cast<uint64_t>(off), bytes, static_cast<char*>(chunks_[c].base) + off};
      return true;
    }
    return false;
  }
  // Returns every pending block whose events have all completed.
  void reclaim() {
    for (auto it = pending_.begin(); it != pending_.end();) {
      bool done = true;
      for (hipEvent_t e : it->events) {
        if (hipEventQuery(e) != hipSuccess) {  // not reached yet (or the query failed: keep the block)
          (void)hipGetLastError();
          done = false;
          break;
        }
      }
      if (!done) {
        ++it;
        continue;
      }
      (void)chunks_[it->block.chunk].alloc.release(it->block.off, it->block.bytes);
      recycle_events(it->events);
      it = pending_.erase(it);
    }
  }
  bool pinned_;
  uint64_t last_size_ = 0;  // size of the newest chunk: the next one doubles it
  std::vector<Chunk> chunks_;
  std::list<Pending> pending_;
  std::vector<hipEvent_t> events_;
};

// Both pools of one device, and the lock that guards them.
struct DevicePools {
  std::mutex mu;
  ListPool dev{false}, pin{true};
};

std::mutex& pools_mu() {
  static std::mutex* mu = new std::mutex();
  return *mu;
}
std::vector<DevicePools*>& all_pools() {
  static std::vector<DevicePools*>* all = new std::vector<DevicePools*>();  // never destroyed
  return *all;
}

DevicePools& pools(int device) {
  std::lock_guard<std::mutex> lock(pools_mu());
  auto& all = all_pools();
  if (device >= static_cast<int>(all.size())) all.resize(device + 1, nullptr);
  if (all[device] == nullptr) all[device] = new DevicePools();
  return *all[device];
}

// After a device-wide synchronisation: gives back the memory of every list no longer held.
void trim_pools_after_sync() {
  std::vector<DevicePools*> all;
  {
    std::lock_guard<std::mutex> lock(pools_mu());
    all = all_pools();
  }
  for (DevicePools* p : all) {
    if (p == nullptr) continue;
    std::lock_guard<std::mutex> lock(p->mu);
    p->dev.trim_after_sync();
    p->pin.trim_after_sync();
  }
}

// Immutable device copies of work lists, keyed by everything that shapes them. Calls hold
// a shared reference from lookup until their launches are enqueued and the launches' event
// is recorded (note_use), so an entry evicted by another thread meanwhile stays alive; when
// the last reference goes, its device block returns to the pool after those events.
struct Plan {
  std::vector<int32_t> cu, cu_loop;  // offsets of the owned and the looped-over segments
  TileRule rule;                     // how block was chosen (part of the key)
  int heads = 0, block = 0, order = 0, device = 0, chunk = 0;
  Item* d_items = nullptr;  // n_items work items, then n_reduce split tiles (loop split)
  int n_items = 0, n_reduce = 0;
  ListPool::Block mem;             // d_items' block in the device pool
  hipEvent_t ready = nullptr;      // upload finished (from the device pool's event pool)
  std::vector<std::pair<hipStream_t, hipEvent_t>> uses;  // last launch reading d_items, per stream
#if T2V_CHECKED
  std::vector<Item> host_items;  // checked builds: the list as uploaded, validated at every call
#endif
  ~Plan() {
    DevicePools& p = pools(device);
    std::lock_guard<std::mutex> lock(p.mu);
    std::vector<hipEvent_t> evs;
    if (ready != nullptr) evs.push_back(ready);
    for (auto& u : uses) evs.push_back(u.second);
    p.dev.release_after(mem, std::move(evs));
  }
};
using PlanRef = std::shared_ptr<Plan>;

// Records, on `stream`, the point after which the launches just enqueued no longer read the
// plan's list. Later launches on the same stream replace the earlier event (stream order).
int note_use(const PlanRef& plan, hipStream_t stream) {
  DevicePools& p = pools(plan->device);
  std::lock_guard<std::mutex> lock(p.mu);
  hipEvent_t ev = nullptr;
  hipError_t e = p.dev.take_event(&ev);
  if (e == hipSuccess) e = hipEventRecord(ev, stream);
  if (e != hipSuccess) {
    if (ev != nullptr) (void)hipEventDestroy(ev);
    // Without the event the list could be reused under a running kernel: keep it alive.
    (void)hipStreamSynchronize(stream);
    return hip_fail(e, "hipEventRecord after launch");
  }
  for (auto& u : plan->uses) {
    if (u.first == stream) {
      std::vector<hipEvent_t> old{u.second};
      p.dev.recycle_events(old);
      u.second = ev;
      return T2V_OK;
    }
  }
  plan->uses.push_back({stream, ev});
  return T2V_OK;
}

constexpr size_t kMaxPlans = 64;

class PlanCache {
 public:
  // Returns the plan (creating and uploading it on `stream` if new) with the
  // upload ordered before any later work on `stream`.
  // The tile rows follow `rule` (chosen once, when the plan is built; plan->block). chunk > 0:
  // the loop split of build_worklist, with the reduce list after the items.
  int get(const int32_t* cu, const int32_t* cu_loop, int nseq, int heads, const TileRule& rule, int order, int chunk,
          hipStream_t stream, PlanRef* out) {
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    std::list<PlanRef> evicted;  // declared before the lock: released after it
    std::lock_guard<std::mutex> lock(mu_);
    for (auto itr = plans_.begin(); itr != plans_.end(); ++itr) {
      Plan& p = **itr;
      if (p.heads == heads && p.rule.same(rule) && p.order == order && p.device == device && p.chunk == chunk &&
          p.cu.size() == static_cast<size_t>(nseq + 1) &&
          std::memcmp(p.cu.data(), cu, sizeof(int32_t) * (nseq + 1)) == 0 &&
          std::memcmp(p.cu_loop.data(), cu_loop, sizeof(int32_t) * (nseq + 1)) == 0) {
        plans_.splice(plans_.begin(), plans_, itr);  // most recently used first
        if (p.ready != nullptr) {
          e = hipStreamWaitEvent(stream, p.ready, 0);
          if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
        }
        *out = *itr;
        return T2V_OK;
      }
    }
    PlanRef p = std::make_shared<Plan>();
    p->cu.assign(cu, cu + nseq + 1);
    p->cu_loop.assign(cu_loop, cu_loop + nseq + 1);
    int ncu = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) {
      (void)hipGetLastError();
      ncu = 0;
    }
    std::vector<Item> items;
    const int block = rule.wide == rule.narrow ? rule.wide
                      : rule.forced == 1       ? rule.wide
                      : rule.forced == 2       ? rule.narrow
                                               : choose_tile_rows(cu, cu_loop, nseq, heads, rule.wide, rule.narrow,
                                                                  rule.narrow_always, rule.max_loop, rule.penalty,
                                                                  order, ncu, &items);
    p->rule = rule;
    p->heads = heads;
    p->block = block;
    p->order = order;
    p->device = device;
    p->chunk = chunk;
    if (items.empty() || chunk > 0) items = build_worklist(cu, cu_loop, nseq, heads, block, order, chunk);
    p->n_items = static_cast<int>(items.size());
    if (chunk > 0) {
      const std::vector<Item> red = build_reduce_list(cu, cu_loop, nseq, heads, block, chunk);
      p->n_reduce = static_cast<int>(red.size());
      items.insert(items.end(), red.begin(), red.end());
    }
    const size_t bytes = items.size() * sizeof(Item);
#if T2V_CHECKED
    p->host_items = items;
#endif
    if (log_enabled()) {
      double ms = 0.0, lb = 0.0;
      plan_makespan(items.data(), p->n_items, block, ncu > 0 ? ncu : 1, &ms, &lb);
      std::fprintf(stderr,
                   "t2v: work list: %d sequences, %d heads, %d-row tiles, %s order: %d items, predicted makespan "
                   "%.4g (lower bound %.4g, ratio %.4f) on %d CUs",
                   nseq, heads, block, order == T2V_ORDER_NATURAL ? "pack" : "longest-first", p->n_items, ms, lb,
                   lb > 0.0 ? ms / lb : 1.0, ncu);
      if (chunk > 0) std::fprintf(stderr, "; loops split at %d rows, %d split tiles", chunk, p->n_reduce);
      std::fprintf(stderr, "\n");
    }
    if (bytes > 0) {
      DevicePools& dp = pools(device);
      std::lock_guard<std::mutex> plock(dp.mu);
      ListPool::Block staging;
      if (int st = dp.dev.alloc(bytes, &p->mem)) return st;
      if (int st = dp.pin.alloc(bytes, &staging)) {
        dp.dev.release_after(p->mem, {});
        p->mem = ListPool::Block{};
        return st;
      }
      p->d_items = static_cast<Item*>(p->mem.ptr);
      std::memcpy(staging.ptr, items.data(), bytes);
      e = hipMemcpyAsync(p->d_items, staging.ptr, bytes, hipMemcpyHostToDevice, stream);
      hipEvent_t copied = nullptr;
      if (e == hipSuccess) e = dp.pin.take_event(&copied);
      if (e == hipSuccess) e = hipEventRecord(copied, stream);
      if (e != hipSuccess) {
        if (copied != nullptr) (void)hipEventDestroy(copied);
        (void)hipStreamSynchronize(stream);  // the staging block may still be read
        dp.pin.release_after(staging, {});
        return hip_fail(e, "upload of the work list");
      }
      dp.pin.release_after(staging, {copied});
      e = dp.dev.take_event(&p->ready);
      if (e == hipSuccess) e = hipEventRecord(p->ready, stream);
      if (e != hipSuccess) return hip_fail(e, "hipEventRecord of the work-list upload");
    }
    plans_.push_front(p);
    *out = p;
    // An evicted plan's list returns to the pool (after its launches) when its last
    // reference goes: here after the lock is released, or later by a call still holding it.
    while (plans_.size() > kMaxPlans) {
      evicted.push_back(std::move(plans_.back()));
      plans_.pop_back();
    }
    return T2V_OK;
  }

  // Waits for the device, then drops every plan and frees the pools' memory.
  void clear() {
    std::list<PlanRef> old;
    {
      std::lock_guard<std::mutex> lock(mu_);
      old.swap(plans_);
    }
    old.clear();  // plans still referenced by a call in progress stay alive until it ends
  }

 private:
  std::mutex mu_;
  std::list<PlanRef> plans_;
};

PlanCache& cache() {
  static PlanCache* c = new PlanCache();  // never destroyed: no HIP calls at process exit
  return *c;
}

#if T2V_CHECKED
// ---------------------------------------------------------------- checked library
//
// Built from the same sources with T2V_CHECKED=1: before any kernel runs, every work list is
// validated on the host against the call's offsets (check_work_items: tile rows against
// cu_seqlens, heads, loop pieces, partial slots); after the launches the call waits for its
// kernels and reads back their device-side DMA row checks. Calls are serialised, since the
// device records belong to the kernel source files, not to calls. A violation returns
// T2V_ERR_BOUNDS naming the list item, or the kernel, workgroup, row and segment length.
std::mutex& checked_mu() {
  static std::mutex m;
  return m;
}

// T2V_CHECK_CANARY=n takes n rows off every bound the kernels check (a correct kernel then
// reports its segments' last rows), to show that the device-side checks report.
unsigned int check_canary() {
  const char* e = std::getenv("T2V_CHECK_CANARY");
  return e != nullptr ? static_cast<unsigned int>(std::max(0, std::atoi(e))) : 0u;
}

int check_list(const std::vector<Item>& items, int n_items, int n_reduce, const int32_t* cu_own,
               const int32_t* cu_loop, int nseq, int heads, int block, int64_t max_slots, const char* kernel) {
  std::string why = check_work_items(items.data(), n_items, cu_own, cu_loop, nseq, heads, block, max_slots, false);
  if (why.empty() && n_reduce > 0)
    why = check_work_items(items.data() + n_items, n_reduce, cu_own, cu_loop, nseq, heads, block, max_slots, true);
  if (!why.empty()) return set_error(T2V_ERR_BOUNDS, std::string("checked library: ") + kernel + " work list, " + why);
  return T2V_OK;
}

int check_plan(const PlanRef& p, const int32_t* cu_own, const int32_t* cu_loop, int nseq, int heads,
               int64_t max_slots, const char* kernel) {
  return check_list(p->host_items, p->n_items, p->n_reduce, cu_own, cu_loop, nseq, heads, p->block, max_slots,
                    kernel);
}

// Set by check_arm once a call is about to launch kernels: only such calls wait for the device
// afterwards (a call refused by validation, or with nothing to do, makes no device call).
thread_local bool t_check_armed = false;

// Clears the kernels' DMA row records and sets the canary, just before a call's first launch.
int check_arm() {
  const unsigned int canary = check_canary();
  unsigned int rec[4];
  for (auto take : {fwd_check_take, dkdv_check_take, dq_check_take}) {
    const hipError_t e = take(rec, canary);
    if (e != hipSuccess) return hip_fail(e, "clearing the DMA row checks");
  }
  t_check_armed = true;
  return T2V_OK;
}

// Waits for this call's kernels, then reports the first DMA row found outside its segment.
int check_collect(hipStream_t s) {
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "waiting for the checked kernels");
  const char* names[3] = {"forward", "dK/dV", "dQ"};
  hipError_t (*takes[3])(unsigned int*, unsigned int) = {fwd_check_take, dkdv_check_take, dq_check_take};
  int status = T2V_OK;
  for (int i = 0; i < 3; ++i) {
    unsigned int rec[4];
    e = takes[i](rec, 0u);
    if (e != hipSuccess) return hip_fail(e, "reading the DMA row checks");
    if (rec[0] != 0u && status == T2V_OK)
      status = set_error(T2V_ERR_BOUNDS, std::string("checked library: ") + names[i] + " kernel, workgroup " +
                                             std::to_string(rec[1]) + " copied row " +
                                             std::to_string(static_cast<int>(rec[2])) + " of a " +
                                             std::to_string(rec[3]) + "-row segment (" + std::to_string(rec[0]) +
                                             " rows outside their segments in this call)");
  }
  return status;
}
#endif

int64_t tensor_bytes(int64_t T, int heads, int head_dim) { return T * heads * head_dim * 2; }

// Optional per-kernel timing: events bracket each launch while enabled.
enum KernelSlot { kSlotFwd = 0, kSlotPre = 1, kSlotDkdv = 2, kSlotDq = 3, kNumSlots = 4 };

class KernelTimer {
 public:
  void set_enabled(bool on) {
    std::lock_guard<std::mutex> lock(mu_);
    drop_locked();
    enabled_ = on;
  }
  // Runs `launch` between two events on `stream` when timing is on.
  template <typename F>
  hipError_t run(int slot, hipStream_t stream, F&& launch) {
    if (!enabled_.load()) return launch();
    hipEvent_t a = nullptr, b = nullptr;
    hipError_t e = hipEventCreate(&a);
    if (e == hipSuccess) e = hipEventCreate(&b);
    if (e == hipSuccess) e = hipEventRecord(a, stream);
    if (e == hipSuccess) e = launch();
    if (e == hipSuccess) e = hipEventRecord(b, stream);
    if (e != hipSuccess) {
      if (a != nullptr) (void)hipEventDestroy(a);
      if (b != nullptr) (void)hipEventDestroy(b);
      return e;
    }
    std::lock_guard<std::mutex> lock(mu_);
    rec_.push_back({slot, a, b});
    return hipSuccess;
  }
  int read(double* ms, int* counts) {
    std::lock_guard<std::mutex> lock(mu_);
    for (int i = 0; i < kNumSlots; ++i) {
      ms[i] = 0.0;
      counts[i] = 0;
    }
    for (const auto& r : rec_) {
      hipError_t e = hipEventSynchronize(r.b);
      float t = 0.0f;
      if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
      if (e != hipSuccess) {
        drop_locked();
        return hip_fail(e, "kernel timing events");
      }
      ms[r.slot] += t;
      counts[r.slot] += 1;
    }
    drop_locked();
    return T2V_OK;
  }

 private:
  struct Rec {
    int slot;
    hipEvent_t a, b;
  };
  void drop_locked() {
    for (const auto& r : rec_) {
      (void)hipEventSynchronize(r.b);
      (void)hipEventDestroy(r.a);
      (void)hipEventDestroy(r.b);
    }
    rec_.clear();
  }
  std::mutex mu_;
  std::atomic<bool> enabled_{false};
  std::vector<Rec> rec_;
};

KernelTimer& timer() {
  static KernelTimer* t = new KernelTimer();
  return *t;
}

// Optional per-workgroup trace: while armed, each MFMA kernel launch takes the next
// n_items records of the caller's buffer (4 uint64 each); a launch that does not fit is
// run untraced and counted as overflowed.
class WorkgroupTracer {
 public:
  void set(unsigned long long* buf, int64_t capacity) {
    std::lock_guard<std::mutex> lock(mu_);
    buf_ = buf;
    cap_ = buf != nullptr ? capacity : 0;
    used_ = 0;
    overflow_ = 0;
  }
  unsigned long long* reserve(int64_t n) {
    std::lock_guard<std::mutex> lock(mu_);
    if (buf_ == nullptr || n <= 0) return nullptr;
    if (used_ + n > cap_) {
      ++overflow_;
      return nullptr;
    }
    unsigned long long* p = buf_ + 4 * used_;
    used_ += n;
    return p;
  }
  void count(int64_t* used, int* overflow) {
    std::lock_guard<std::mutex> lock(mu_);
    *used = used_;
    *overflow = overflow_;
  }

 private:
  std::mutex mu_;
  unsigned long long* buf_ = nullptr;
  int64_t cap_ = 0, used_ = 0;
  int overflow_ = 0;
};

WorkgroupTracer& tracer() {
  static WorkgroupTracer* t = new WorkgroupTracer();
  return *t;
}

}  // namespace
}  // namespace t2v

namespace t2v {
namespace {

// Forward over queries at cu_q and keys at cu_k (the same array for self-attention).
int attn_fwd_impl(const void* q, const void* k, const void* v, const int32_t* cu_q, const int32_t* cu_k, int nseq,
                  int heads, int head_dim, float scale, void* out, float* lse, void* stream) {
  if (int st = check_offsets_on_host(cu_q, cu_k)) return st;
  int64_t Tq = 0, Tk = 0;
  if (cu_q == cu_k) {
    if (int st = validate_shape(cu_q, nseq, heads, head_dim, scale, &Tq)) return st;
    Tk = Tq;
  } else if (int st = validate_shape_qk(cu_q, cu_k, nseq, heads, head_dim, scale, &Tq, &Tk)) {
    return st;
  }
  if (Tq == 0) return T2V_OK;
  const int64_t qb = tensor_bytes(Tq, heads, head_dim), kb = tensor_bytes(Tk, heads, head_dim);
  const int64_t lb = Tq * heads * 4;
  if (int st = validate_pointers({{q, qb, "q"}, {k, kb, "k"}, {v, kb, "v"}}, {{out, qb, "out"}, {lse, lb, "lse"}}))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  PlanRef plan;
  if (int st = cache().get(cu_q, cu_k, nseq, heads, fwd_rule(head_dim), order_from_env(), 0, s, &plan)) return st;
#if T2V_CHECKED
  if (int st = check_plan(plan, cu_q, cu_k, nseq, heads, 0, "forward")) return st;
#endif
  if (plan->n_items == 0) return T2V_OK;
#if T2V_CHECKED
  if (int st = check_arm()) return st;
#endif
  AttnArgs a{};
  a.q_rows = plan->block;
  a.q = q;
  a.k = k;
  a.v = v;
  a.heads = heads;
  a.head_dim = head_dim;
  a.total_tokens = Tq;
  a.scale = scale;
  a.trace = tracer().reserve(plan->n_items);
  a.persistent = persistent_enabled();
  hipError_t e = timer().run(kSlotFwd, s, [&] { return launch_fwd(a, out, lse, plan->d_items, plan->n_items, s); });
  const int used = note_use(plan, s);
  if (e != hipSuccess) return hip_fail(e, "forward kernel launch");
  return used;
}

int attn_bwd_impl(const void* q, const void* k, const void* v, const void* out, const float* lse, const int32_t* cu_q,
                  const int32_t* cu_k, int nseq, int heads, int head_dim, float scale, const void* dout, void* dq,
                  void* dk, void* dv, float* delta_ws, void* stream) {
  if (int st = check_offsets_on_host(cu_q, cu_k)) return st;
  int64_t Tq = 0, Tk = 0;
  if (cu_q == cu_k) {
    if (int st = validate_shape(cu_q, nseq, heads, head_dim, scale, &Tq)) return st;
    Tk = Tq;
  } else if (int st = validate_shape_qk(cu_q, cu_k, nseq, heads, head_dim, scale, &Tq, &Tk)) {
    return st;
  }
  if (Tq == 0) return T2V_OK;
  const int64_t qb = tensor_bytes(Tq, heads, head_dim), kb = tensor_bytes(Tk, heads, head_dim);
  const int64_t lb = Tq * heads * 4;
  if (int st = validate_pointers(
          {{q, qb, "q"}, {k, kb, "k"}, {v, kb, "v"}, {out, qb, "out"}, {lse, lb, "lse"}, {dout, qb, "dout"}},
          {{dq, qb, "dq"}, {dk, kb, "dk"}, {dv, kb, "dv"}, {delta_ws, 2 * lb, "delta_ws"}}))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int order = order_from_env();
  PlanRef pk, pq;
  // dK/dV tiles own keys and loop over queries; dQ tiles own queries and loop over keys.
  // Loops too long for the available parallelism (short keys, long queries) are split into
  // pieces whose fp32 partial sums go to slots in dq's memory: dq is an output that the dQ
  // kernel, launched after the reduce, overwrites, so the slots are capped at its size.
  const int kv_rows = dkdv_tile_rows(head_dim);
  int chunk = 0;
  if (split_enabled())
    chunk = choose_loop_split(cu_k, cu_q, nseq, heads, kv_rows, cu_count(), qb / dkdv_partial_slot_bytes(head_dim))
                .chunk;
  if (int st = cache().get(cu_k, cu_q, nseq, heads, dkdv_rule(head_dim), order, chunk, s, &pk)) return st;
  if (int st = cache().get(cu_q, cu_k, nseq, heads, dq_rule(head_dim), order, 0, s, &pq)) return st;
#if T2V_CHECKED
  if (int st = check_plan(pk, cu_k, cu_q, nseq, heads, qb / dkdv_partial_slot_bytes(head_dim), "dK/dV")) return st;
  if (int st = check_plan(pq, cu_q, cu_k, nseq, heads, 0, "dQ")) return st;
#endif
  AttnArgs a{};
  a.q_rows = pq->block;
  a.partial = static_cast<float*>(dq);
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.dout = dout;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.delta = delta_ws;
  a.heads = heads;
  a.head_dim = head_dim;
  a.total_tokens = Tq;
  a.scale = scale;
  a.persistent = persistent_enabled();
#if T2V_CHECKED
  if (int st = check_arm()) return st;
#endif
  hipError_t e = timer().run(kSlotPre, s, [&] { return launch_bwd_pre(a, s); });
  if (e != hipSuccess) return hip_fail(e, "backward preprocess launch");
  if (pk->n_items > 0) {
    a.trace = tracer().reserve(pk->n_items);
    e = timer().run(kSlotDkdv, s, [&] {
      hipError_t r = launch_bwd_dkdv(a, pk->d_items, pk->n_items, s);
      if (r == hipSuccess && pk->n_reduce > 0) r = launch_bwd_dkdv_reduce(a, pk->d_items + pk->n_items, pk->n_reduce, s);
      return r;
    });
    const int used = note_use(pk, s);
    if (e != hipSuccess) return hip_fail(e, "dK/dV kernel launch");
    if (used != T2V_OK) return used;
  }
  if (pq->n_items > 0) {
    a.trace = tracer().reserve(pq->n_items);
    e = timer().run(kSlotDq, s, [&] { return launch_bwd_dq(a, pq->d_items, pq->n_items, s); });
    const int used = note_use(pq, s);
    if (e != hipSuccess) return hip_fail(e, "dQ kernel launch");
    if (used != T2V_OK) return used;
  }
  return T2V_OK;
}

// ------------------------------------------------------------ backward without allocation
//
// For callers that cannot allocate device memory: the [2, H, T] Delta / lse scratch and
// both work lists live in one static device array, `scratch`, instead of the caller's
// delta_ws and the library's list pool. Its device address is taken once per GPU (with
// that GPU current) and kept; host code uses only that address, never the array's name.
// Every call on a GPU shares the array, so calls that overlap on one GPU (different
// streams, or threads) race; calls on one stream are ordered by it. Nothing in it needs
// to start at zero: each call overwrites the parts it reads (the Delta pass writes the
// scratch rows, the list uploads the items).
constexpr size_t kScratchAlign = 256;

size_t align_up(size_t n) { return (n + kScratchAlign - 1) / kScratchAlign * kScratchAlign; }

int scratch_address(int device, unsigned char** out) {
  static std::mutex* mu = new std::mutex();
  static std::vector<unsigned char*>* ptrs = new std::vector<unsigned char*>();  // never destroyed
  std::lock_guard<std::mutex> lock(*mu);
  if (device >= static_cast<int>(ptrs->size())) ptrs->resize(device + 1, nullptr);
  if ((*ptrs)[device] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return set_error(T2V_ERR_HIP, std::string("hipGetSymbolAddress of the no-allocation scratch: ") +
                                        hipGetErrorString(e));
    }
    (*ptrs)[device] = static_cast<unsigned char*>(p);
  }
  *out = (*ptrs)[device];
  return T2V_OK;
}

int attn_bwd_noalloc_impl(const void* q, const void* k, const void* v, const void* out, const float* lse,
                          const int32_t* cu, int nseq, int heads, int head_dim, float scale, const void* dout,
                          void* dq, void* dk, void* dv, void* stream) {
  if (int st = check_offsets_on_host(cu, cu)) return st;
  int64_t T = 0;
  if (int st = validate_shape(cu, nseq, heads, head_dim, scale, &T)) return st;
  if (T == 0) return T2V_OK;
  const int64_t tb = tensor_bytes(T, heads, head_dim), lb = T * heads * 4;
  if (int st = validate_pointers(
          {{q, tb, "q"}, {k, tb, "k"}, {v, tb, "v"}, {out, tb, "out"}, {lse, lb, "lse"}, {dout, tb, "dout"}},
          {{dq, tb, "dq"}, {dk, tb, "dk"}, {dv, tb, "dv"}}))
    return st;
  const size_t delta_bytes = align_up(static_cast<size_t>(2 * lb));
  auto too_big = [&](size_t need) {
    return set_error(T2V_ERR_INVALID_ARG,
                     "the no-allocation backward needs " + std::to_string(need) + " bytes of scratch (8 * heads * T "
                     "for Delta and lse, 32 per work item), more than its " +
                     std::to_string(kNoAllocScratchBytes) + "-byte array");
  };
  if (delta_bytes > kNoAllocScratchBytes) return too_big(delta_bytes);
  // The same work lists as t2v_attn_bwd (tile rules, order, loop split), built per call.
  const int order = order_from_env();
  const int kv_rows = dkdv_tile_rows(head_dim);
  const int ncu = cu_count();
  int chunk = 0;
  if (split_enabled()) chunk = choose_loop_split(cu, cu, nseq, heads, kv_rows, ncu, tb / dkdv_partial_slot_bytes(head_dim)).chunk;
  std::vector<Item> kv = build_worklist(cu, cu, nseq, heads, kv_rows, order, chunk);
  const int n_kv = static_cast<int>(kv.size());
  int n_reduce = 0;
  if (chunk > 0) {
    const std::vector<Item> red = build_reduce_list(cu, cu, nseq, heads, kv_rows, chunk);
    n_reduce = static_cast<int>(red.size());
    kv.insert(kv.end(), red.begin(), red.end());
  }
  const TileRule qr = dq_rule(head_dim);
  std::vector<Item> ql;
  const int q_rows = qr.forced == 1   ? qr.wide
                     : qr.forced == 2 ? qr.narrow
                                      : choose_tile_rows(cu, cu, nseq, heads, qr.wide, qr.narrow, qr.narrow_always,
                                                         qr.max_loop, qr.penalty, order, ncu, &ql);
  if (ql.empty()) ql = build_worklist(cu, cu, nseq, heads, q_rows, order);
#if T2V_CHECKED
  if (int st = check_list(kv, n_kv, n_reduce, cu, cu, nseq, heads, kv_rows, tb / dkdv_partial_slot_bytes(head_dim),
                          "dK/dV"))
    return st;
  if (int st = check_list(ql, static_cast<int>(ql.size()), 0, cu, cu, nseq, heads, q_rows, 0, "dQ")) return st;
#endif
  const size_t kv_bytes = align_up(kv.size() * sizeof(Item)), q_bytes = align_up(ql.size() * sizeof(Item));
  if (delta_bytes + kv_bytes + q_bytes > kNoAllocScratchBytes) return too_big(delta_bytes + kv_bytes + q_bytes);
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  unsigned char* base = nullptr;
  if (int st = scratch_address(device, &base)) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Item* d_kv = reinterpret_cast<Item*>(base + delta_bytes);
  Item* d_q = reinterpret_cast<Item*>(base + delta_bytes + kv_bytes);
  // Pageable sources: the runtime stages them itself, in stream order (the call returns once
  // the host arrays may be released).
  if (!kv.empty()) e = hipMemcpyAsync(d_kv, kv.data(), kv.size() * sizeof(Item), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !ql.empty()) e = hipMemcpyAsync(d_q, ql.data(), ql.size() * sizeof(Item), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "upload of the work lists into the no-allocation scratch");
  AttnArgs a{};
  a.q_rows = q_rows;
  a.partial = static_cast<float*>(dq);
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.dout = dout;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.delta = reinterpret_cast<float*>(base);
  a.heads = heads;
  a.head_dim = head_dim;
  a.total_tokens = T;
  a.scale = scale;
  a.persistent = persistent_enabled();
#if T2V_CHECKED
  if (int st = check_arm()) return st;
#endif
  e = timer().run(kSlotPre, s, [&] { return launch_bwd_pre(a, s); });
  if (e != hipSuccess) return hip_fail(e, "backward preprocess launch");
  if (n_kv > 0) {
    a.trace = tracer().reserve(n_kv);
    e = timer().run(kSlotDkdv, s, [&] {
      hipError_t r = launch_bwd_dkdv(a, d_kv, n_kv, s);
      if (r == hipSuccess && n_reduce > 0) r = launch_bwd_dkdv_reduce(a, d_kv + n_kv, n_reduce, s);
      return r;
    });
    if (e != hipSuccess) return hip_fail(e, "dK/dV kernel launch");
  }
  if (!ql.empty()) {
    a.trace = tracer().reserve(static_cast<int64_t>(ql.size()));
    e = timer().run(kSlotDq, s, [&] { return launch_bwd_dq(a, d_q, static_cast<int>(ql.size()), s); });
    if (e != hipSuccess) return hip_fail(e, "dQ kernel launch");
  }
  return T2V_OK;
}

// Runs f, turning host exceptions into statuses (none may cross the C ABI).
template <typename F>
int guarded(F&& f) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return set_error(T2V_ERR_OOM, "host allocation failed");
  } catch (...) {
    return set_error(T2V_ERR_INVALID_ARG, "unexpected host exception");
  }
}

// Runs an attention call; in the checked library, serialised and followed by the kernels'
// device-side checks.
template <typename F>
int checked_call(void* stream, F&& f) {
#if T2V_CHECKED
  std::lock_guard<std::mutex> lock(checked_mu());
  t_check_armed = false;
  const int st = f();
  if (st != T2V_OK || !t_check_armed) return st;
  t_check_armed = false;
  return check_collect(static_cast<hipStream_t>(stream));
#else
  (void)stream;
  return f();
#endif
}

}  // namespace
}  // namespace t2v

namespace t2v {

int persistent_grid(const void* kernel, int threads, int n_items) {
  int per_cu = 0, ncu = cu_count();
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) {
    (void)hipGetLastError();
    per_cu = 1;
  }
  int grid = std::max(1, per_cu) * std::max(1, ncu);
  if (grid >= kNumXcd) grid -= grid % kNumXcd;
  return std::max(1, std::min(grid, n_items));
}

}  // namespace t2v

extern "C" {

int t2v_attn_fwd(const void* q, const void* k, const void* v, const int32_t* cu_seqlens, int nseq, int heads,
                 int head_dim, float scale, void* out, float* lse, void* stream) {
  return t2v::guarded([&] {
    return t2v::checked_call(stream, [&] {
      return t2v::attn_fwd_impl(q, k, v, cu_seqlens, cu_seqlens, nseq, heads, head_dim, scale, out, lse, stream);
    });
  });
}

int t2v_attn_bwd(const void* q, const void* k, const void* v, const void* out, const float* lse,
                 const int32_t* cu_seqlens, int nseq, int heads, int head_dim, float scale, const void* dout,
                 void* dq, void* dk, void* dv, float* delta_ws, void* stream) {
  return t2v::guarded([&] {
    return t2v::checked_call(stream, [&] {
      return t2v::attn_bwd_impl(q, k, v, out, lse, cu_seqlens, cu_seqlens, nseq, heads, head_dim, scale, dout, dq,
                                dk, dv, delta_ws, stream);
    });
  });
}

int t2v_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* out, const float* lse,
                         const int32_t* cu_seqlens, int nseq, int heads, int head_dim, float scale, const void* dout,
                         void* dq, void* dk, void* dv, void* stream) {
  return t2v::guarded([&] {
    return t2v::checked_call(stream, [&] {
      return t2v::attn_bwd_noalloc_impl(q, k, v, out, lse, cu_seqlens, nseq, heads, head_dim, scale, dout, dq, dk,
                                        dv, stream);
    });
  });
}

int t2v_attn_fwd_qk(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_q,
                    const int32_t* cu_seqlens_k, int nseq, int heads, int head_dim, float scale, void* out, float* lse,
                    void* stream) {
  return t2v::guarded([&] {
    if (cu_seqlens_q == nullptr || cu_seqlens_k == nullptr)
      return t2v::set_error(T2V_ERR_INVALID_ARG, "cu_seqlens_q or cu_seqlens_k is NULL");
    return t2v::checked_call(stream, [&] {
      return t2v::attn_fwd_impl(q, k, v, cu_seqlens_q, cu_seqlens_k, nseq, heads, head_dim, scale, out, lse, stream);
    });
  });
}

int t2v_attn_bwd_qk(const void* q, const void* k, const void* v, const void* out, const float* lse,
                    const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int nseq, int heads, int head_dim,
                    float scale, const void* dout, void* dq, void* dk, void* dv, float* delta_ws, void* stream) {
  return t2v::guarded([&] {
    if (cu_seqlens_q == nullptr || cu_seqlens_k == nullptr)
      return t2v::set_error(T2V_ERR_INVALID_ARG, "cu_seqlens_q or cu_seqlens_k is NULL");
    return t2v::checked_call(stream, [&] {
      return t2v::attn_bwd_impl(q, k, v, out, lse, cu_seqlens_q, cu_seqlens_k, nseq, heads, head_dim, scale, dout,
                                dq, dk, dv, delta_ws, stream);
    });
  });
}

int t2v_timing_enable(int on) {
  t2v::timer().set_enabled(on != 0);
  return T2V_OK;
}

int t2v_kernel_times(double* ms_out, int* counts_out) {
  if (ms_out == nullptr || counts_out == nullptr) return t2v::set_error(T2V_ERR_INVALID_ARG, "NULL output");
  return t2v::timer().read(ms_out, counts_out);
}

int t2v_trace_set(unsigned long long* dev_records, int64_t capacity) {
  if (capacity < 0 || (dev_records == nullptr && capacity != 0))
    return t2v::set_error(T2V_ERR_INVALID_ARG, "capacity must be >= 0, and 0 when dev_records is NULL");
  if (dev_records != nullptr && reinterpret_cast<uintptr_t>(dev_records) % 8 != 0)
    return t2v::set_error(T2V_ERR_INVALID_ARG, "dev_records is not 8-byte aligned");
  t2v::tracer().set(dev_records, capacity);
  return T2V_OK;
}

int t2v_trace_count(int64_t* n_records, int* n_overflowed) {
  if (n_records == nullptr || n_overflowed == nullptr) return t2v::set_error(T2V_ERR_INVALID_ARG, "NULL output");
  t2v::tracer().count(n_records, n_overflowed);
  return T2V_OK;
}

void t2v_release_cache(void) {
  (void)hipDeviceSynchronize();
  t2v::cache().clear();
  t2v::trim_pools_after_sync();
}

}  // extern "C"
