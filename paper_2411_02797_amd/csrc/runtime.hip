// Host runtime of libcct: argument checks, the tree handle, a caching device-memory
// pool, and the orchestration of ingest -> publish -> canonical ordering -> emission
// on the caller's stream.  See include/cct.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "cct.h"
#include "common.h"

using namespace cct;

namespace {

// message of the calling thread's last failure: a fixed buffer, so that reporting an
// error never allocates
thread_local char g_error[256];
thread_local double g_timings[5] = {0, 0, 0, 0, 0};
thread_local double g_join_ms = 0;  // correlation-ID join of the last cct_merge_activity
thread_local double g_view_ms = 0;  // the most recent computation of a bottom-up view
thread_local double g_filter_ms = 0;  // the last cct_filter
thread_local double g_stats_ms = 0;   // statistics kept by the last build/merge (0 without)
thread_local double g_node_stats_ms = 0;  // the last cct_stats
thread_local double g_query_ms = 0;       // the last cct_query's lookups
thread_local double g_qindex_ms = 0;      // the prefix index built by the last cct_query (0 if kept)
thread_local int g_alloc_countdown = 0;  // test hook: >0 makes the n-th allocation of a call fail

int64_t env_int(const char *name, int64_t dflt) {
  const char *v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::strtoll(v, nullptr, 10);
}

cct_status fail(cct_status s, const char *msg) {
  std::snprintf(g_error, sizeof g_error, "%s", msg);
  return s;
}
void clear_error() { g_error[0] = 0; }

// Arms the test hook for one public call (CCT_TEST_FAIL_ALLOC = n: the call's n-th pool
// allocation fails) and disarms it when the call returns, so no count carries over into
// the next call.
struct AllocHook {
  AllocHook() { g_alloc_countdown = (int)env_int("CCT_TEST_FAIL_ALLOC", 0); }
  ~AllocHook() { g_alloc_countdown = 0; }
};

// ---- caching device-memory pool --------------------------------------------------
struct Pool {
  std::mutex mu;
  std::multimap<std::pair<int, size_t>, void *> cache;  // (device, bytes) -> block
  std::unordered_map<void *, std::pair<int, size_t>> live;
};
Pool &pool() {
  static Pool *p = new Pool;  // never destroyed: blocks may outlive static destructors
  return *p;
}

size_t round_bytes(size_t b) {
  if (b < 256) return 256;
  if (b < (1u << 20)) return (b + 255) & ~(size_t)255;
  return (b + (1u << 20) - 1) & ~(size_t)((1u << 20) - 1);
}

void *pool_alloc(size_t bytes) {
  if (g_alloc_countdown > 0 && --g_alloc_countdown == 0) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  const size_t want = round_bytes(bytes);
  Pool &P = pool();
  {
    std::lock_guard<std::mutex> lk(P.mu);
    auto it = P.cache.lower_bound({dev, want});
    if (it != P.cache.end() && it->first.first == dev && it->first.second <= 2 * want) {
      void *p = it->second;
      P.live[p] = it->first;
      P.cache.erase(it);
      return p;
    }
  }
  void *p = nullptr;
  if (hipMalloc(&p, want) != hipSuccess) {
    (void)hipGetLastError();
    cct_release_cached_memory();
    if (hipMalloc(&p, want) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
  }
  std::lock_guard<std::mutex> lk(P.mu);
  P.live[p] = {dev, want};
  return p;
}

void pool_free(void *p) {
  if (!p) return;
  Pool &P = pool();
  std::lock_guard<std::mutex> lk(P.mu);
  auto it = P.live.find(p);
  if (it == P.live.end()) return;
  P.cache.emplace(it->second, p);
  P.live.erase(it);
}

// An owned device buffer from the pool.
struct Buf {
  void *p = nullptr;
  size_t bytes = 0;
  Buf() = default;
  Buf(const Buf &) = delete;
  Buf &operator=(const Buf &) = delete;
  Buf(Buf &&o) noexcept : p(o.p), bytes(o.bytes) { o.p = nullptr; o.bytes = 0; }
  Buf &operator=(Buf &&o) noexcept {
    if (this != &o) { release(); p = o.p; bytes = o.bytes; o.p = nullptr; o.bytes = 0; }
    return *this;
  }
  ~Buf() { release(); }
  bool alloc(size_t n) {
    release();
    p = pool_alloc(n ? n : 1);
    bytes = p ? n : 0;
    return p != nullptr;
  }
  void release() { pool_free(p); p = nullptr; bytes = 0; }
  template <class T> T *as() const { return static_cast<T *>(p); }
};

int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    hipDeviceProp_t prop;
    cached[dev] = hipGetDeviceProperties(&prop, dev) == hipSuccess ? prop.multiProcessorCount : 256;
  }
  return cached[dev];
}

// pinned host staging for small device -> host reads
unsigned long long *host_scratch() {
  thread_local unsigned long long *h = nullptr;
  if (!h && hipHostMalloc((void **)&h, 64 * sizeof(unsigned long long), hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();
    h = nullptr;
  }
  return h;
}

// Second streams for work that overlaps the caller's stream within one call (default
// priority, non-blocking: ordered only by the events the call records).  A call takes one
// from its device's pool and gives it back when it returns, so concurrent calls on other
// trees never share one.
struct StreamPool {
  std::mutex mu;
  std::vector<std::pair<int, hipStream_t>> free;  // (device, stream)
};
StreamPool &stream_pool() {
  static StreamPool *p = new StreamPool;  // never destroyed: streams live until the process ends
  return *p;
}

// Holds a side stream for one call; on return it waits for the stream (before the
// buffers its work uses are released: declare it after them) and gives it back.
struct SideGuard {
  hipStream_t st = nullptr;
  int dev = 0;
  hipStream_t acquire() {
    if (hipGetDevice(&dev) != hipSuccess) { (void)hipGetLastError(); return nullptr; }
    StreamPool &P = stream_pool();
    {
      std::lock_guard<std::mutex> lock(P.mu);
      for (size_t i = 0; i < P.free.size(); ++i)
        if (P.free[i].first == dev) {
          st = P.free[i].second;
          P.free.erase(P.free.begin() + (long)i);
          return st;
        }
    }
    if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) {
      (void)hipGetLastError();
      st = nullptr;
    }
    return st;
  }
  ~SideGuard() {
    if (!st) return;
    (void)hipStreamSynchronize(st);
    StreamPool &P = stream_pool();
    std::lock_guard<std::mutex> lock(P.mu);
    P.free.emplace_back(dev, st);
  }
};

// Wait for the work queued on s so far by polling an event (the host spins; a blocking
// wait adds its wake-up latency to the call's critical path).
hipError_t spin_sync(hipStream_t s) {
  hipEvent_t e = nullptr;
  hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
  if (r != hipSuccess) return hipStreamSynchronize(s);
  r = hipEventRecord(e, s);
  if (r == hipSuccess) {
    while ((r = hipEventQuery(e)) == hipErrorNotReady) {
    }
  }
  (void)hipEventDestroy(e);
  return r;
}

// An event for ordering two streams (no timing).
struct Event {
  hipEvent_t ev = nullptr;
  Event() {
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) { (void)hipGetLastError(); ev = nullptr; }
  }
  ~Event() {
    if (ev) (void)hipEventDestroy(ev);
  }
};

uint64_t pow2_at_least(uint64_t x) {
  uint64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

int floor_log2(uint64_t x) {
  int l = 0;
  while ((x >> 1) >= 1 && x > 1) { x >>= 1; ++l; }
  return l;
}

}  // namespace

// ---- the tree ------------------------------------------------------------------------
struct cct_tree {
  int device = 0;
  int32_t m = 1;
  // unique-path table (slot words); sums live per path in psums
  uint64_t cap = 0;
  Buf slot;
  // path store
  int64_t d = 0, dcap = 0;
  int64_t store_used = 0, store_cap = 0, sum_len = 0;
  Buf pframes, pcp, pstart, plen, pslot, psums;
  // per-path statistics (count, minima, sums of squares), kept when built with them
  bool stats = false;
  Buf pcnt, pmin, psq;
  // canonical arrays
  int64_t u = 0;
  Buf parent, frame, depth, subend, excl, incl;
  // bottom-up view (cct_bottom_up), kept until the tree changes; bu_k < 0: not computed
  int64_t bu_k = -1;
  Buf bu_frames, bu_excl, bu_incl;
  // query index, built by the first cct_query and kept until the tree changes (mutable: a
  // query leaves the tree itself as it is)
  mutable bool q_ready = false;
  mutable uint64_t q_cap = 0, q_hash_mask = 0;  // q_cap = 0: no index (binary search)
  mutable Buf q_sorted, q_tab;
  // canonical metadata kept for queries
  Buf order, lcp, scan_out;
};

namespace {

#define HIP_TRY(x)                                              \
  do {                                                          \
    hipError_t e_ = (x);                                        \
    if (e_ != hipSuccess) {                                     \
      (void)hipGetLastError();                                  \
      return fail(CCT_EDEVICE, hipGetErrorString(e_));          \
    }                                                           \
  } while (0)

cct_status check_paths(const cct_paths *p, bool need_metrics) {
  if (!p) return fail(CCT_EINVAL, "paths is NULL");
  if (p->n_events < 0 || p->n_frames < 0) return fail(CCT_EINVAL, "negative size");
  if (p->n_events > CCT_MAX_EVENTS) return fail(CCT_EOVERFLOW, "too many events in one call");
  if (p->n_metrics < 1 || p->n_metrics > CCT_MAX_METRICS) return fail(CCT_EINVAL, "n_metrics out of range");
  if (!p->offsets) return fail(CCT_EINVAL, "offsets is NULL");
  if (p->n_frames > 0 && !p->frames) return fail(CCT_EINVAL, "frames is NULL");
  if (need_metrics && p->n_events > 0 && !p->metrics) return fail(CCT_EINVAL, "metrics is NULL");
  if (((uintptr_t)p->offsets & 7) || ((uintptr_t)p->frames & 3) || ((uintptr_t)p->metrics & 7))
    return fail(CCT_EINVAL, "misaligned pointer");
  return CCT_OK;
}

// Grow a device array to hold `need` bytes, keeping the first `keep` bytes.
cct_status grow(Buf &b, size_t need, size_t keep, hipStream_t s) {
  if (b.p && b.bytes >= need) return CCT_OK;
  Buf nb;
  if (!nb.alloc(need)) return fail(CCT_ENOMEM, "device allocation failed");
  if (keep) HIP_TRY(hipMemcpyAsync(nb.p, b.p, keep, hipMemcpyDeviceToDevice, s));
  b = std::move(nb);
  return CCT_OK;
}

// HIP events on the call's stream: 0 call start, 1/2 around the ingest kernel, 3 after
// publish, 4 after the sort, 5 after node emission.
struct Timer {
  hipEvent_t ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  bool ok = true;
  Timer() {
    for (auto &e : ev)
      if (hipEventCreate(&e) != hipSuccess) { ok = false; (void)hipGetLastError(); }
  }
  ~Timer() {
    for (auto &e : ev)
      if (e) (void)hipEventDestroy(e);
  }
  void mark(int i, hipStream_t s) {
    if (ok) (void)hipEventRecord(ev[i], s);
  }
  float span(int a, int b) {
    float ms = 0;
    if (hipEventElapsedTime(&ms, ev[a], ev[b]) != hipSuccess) { (void)hipGetLastError(); return 0; }
    return ms;
  }
  // timings: ingest kernel, publish, sort, emission, whole call
  void collect(bool ingested) {
    for (int i = 0; i < 5; ++i) g_timings[i] = 0;
    if (!ok) return;
    if (ingested) g_timings[0] = span(1, 2);
    g_timings[1] = span(2, 3);
    g_timings[2] = span(3, 4);
    g_timings[3] = span(4, 5);
    g_timings[4] = span(0, 5);
  }
};

// Staging of the metric aggregation (launch_aggregate) for `n_rows` rows keyed by slots
// below `cap`: bucket counts zeroed on `s`.  Leaves st.nbuckets = 0 (atomic flush) when
// the slots need more buckets than a workgroup can count.
cct_status setup_stage(int32_t m, uint64_t cap, int agg_grid, Buf &count, Buf &keys, Buf &sums, AggStage &st,
                       hipStream_t s) {
  st = AggStage{};
  st.bshift = agg_bucket_shift(m);
  const int64_t nbk = std::max<int64_t>(1, (int64_t)((cap + (1ull << st.bshift) - 1) >> st.bshift));
  if (nbk > agg_max_buckets()) return CCT_OK;
  const int64_t total = (int64_t)agg_grid * agg_map_entries(m);
  st.nbuckets = nbk;
  st.bucket_cap = 2 * ((total + nbk - 1) / nbk) + 256;  // twice the even share (slots are hashed)
  if (!count.alloc(nbk * 4) || !keys.alloc(nbk * st.bucket_cap * 4) || !sums.alloc(nbk * st.bucket_cap * m * 8))
    return fail(CCT_ENOMEM, "device allocation failed");
  HIP_TRY(hipMemsetAsync(count.p, 0, nbk * 4, s));
  st.count = count.as<uint32_t>();
  st.keys = keys.as<uint32_t>();
  st.sums = sums.as<uint64_t>();
  return CCT_OK;
}

// Re-insert the tree's stored paths into a fresh table of capacity `cap`.  Both new
// arrays are allocated before any work is queued, and the stream is synchronised before
// the old table and slot list go back to the pool (work queued earlier may still read
// them; a pool block must be idle before it can be handed out again).
cct_status rehash(cct_tree *t, uint64_t cap, uint64_t hash_mask, hipStream_t s) {
  Buf ns, np;
  if (!ns.alloc(cap * sizeof(Slot)) || (t->d > 0 && !np.alloc(t->dcap * 4)))
    return fail(CCT_ENOMEM, "device allocation failed");
  hipError_t e = hipMemsetAsync(ns.p, 0xFF, cap * sizeof(Slot), s);
  if (e == hipSuccess && t->d > 0) {
    launch_rehash(t->pframes.as<uint32_t>(), t->pstart.as<int64_t>(), t->plen.as<uint32_t>(), t->d,
                  ns.as<Slot>(), cap - 1, hash_mask, np.as<uint32_t>(), s);
    e = hipGetLastError();
  }
  const hipError_t es = hipStreamSynchronize(s);
  if (e == hipSuccess) e = es;
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(CCT_EDEVICE, hipGetErrorString(e));
  }
  if (t->d > 0) t->pslot = std::move(np);
  t->slot = std::move(ns);
  t->cap = cap;
  return CCT_OK;
}

// Aggregate one batch into `t` (fresh or existing).  Strong guarantee: on error the
// tree's table, path store, sums and node arrays are as before.  Every array the call
// changes is either new (sums and statistics are folded into fresh copies, swapped in
// at the commit) or changed only past the part the tree uses (path store entries of new
// paths); what the call puts into the table (claims, then the published slots) is
// taken out again on the failure path.
cct_status aggregate(cct_tree *t, const cct_paths *p, hipStream_t s) {
  const int32_t m = t->m;
  const int64_t N = p->n_events;
  const int hash_bits = (int)env_int("CCT_TEST_HASH_BITS", 64);
  const uint64_t hash_mask = hash_bits >= 64 ? ~0ull : ((1ull << (hash_bits < 0 ? 0 : hash_bits)) - 1);
  unsigned long long *hs = host_scratch();
  if (!hs) return fail(CCT_ENOMEM, "pinned host allocation failed");
  Timer tm;
  tm.mark(0, s);

  Buf ctr;
  if (!ctr.alloc(kCtrCount * 8 + 64)) return fail(CCT_ENOMEM, "device allocation failed");
  unsigned long long *dctr = ctr.as<unsigned long long>();

  // Failure path: this call's claims (before they are published) or its published slots
  // are emptied again, and both of the call's streams are synchronised before any of its
  // buffers returns to the pool (a pool block must be idle before it is handed out).
  Buf new_slots;
  uint64_t n_new = 0;
  bool claimed = false, published = false;
  hipStream_t side = s;
  auto undo = [&](cct_status st) -> cct_status {
    if (published) launch_reset_slots(t->slot.as<Slot>(), new_slots.as<uint32_t>(), (int64_t)n_new, s);
    else if (claimed) launch_unclaim(t->slot.as<Slot>(), t->cap, s);
    (void)hipGetLastError();
    (void)hipStreamSynchronize(s);
    if (side != s) (void)hipStreamSynchronize(side);
    return st;
  };
#define AGG_TRY(x)                                              \
  do {                                                          \
    hipError_t e_ = (x);                                        \
    if (e_ != hipSuccess) {                                     \
      (void)hipGetLastError();                                  \
      return undo(fail(CCT_EDEVICE, hipGetErrorString(e_)));    \
    }                                                           \
  } while (0)

  if (N == 0) {
    // nothing to insert; offsets[0] must still be 0 and n_frames 0
    if (p->n_frames != 0) return fail(CCT_EINVAL, "n_frames != offsets[N]");
    AGG_TRY(hipMemcpyAsync(hs, p->offsets, 8, hipMemcpyDeviceToHost, s));
    AGG_TRY(hipStreamSynchronize(s));
    if (hs[0] != 0) return fail(CCT_EINVAL, "offsets[0] != 0");
    if (t->parent.p) return CCT_OK;
    tm.mark(1, s);
    tm.mark(2, s);
  }

  // ---- A1-A3: ingest (retry with a larger table on overflow) -------------------------
  // keep the table at most half full before inserting
  if ((uint64_t)t->d * 2 > t->cap) {
    cct_status st = rehash(t, pow2_at_least((uint64_t)t->d * 4), hash_mask, s);
    if (st) return st;
  }
  Buf delta, slot_of, cpart, agg_count, agg_keys, agg_sums, nlen, nsrc;
  uint64_t new_frames = 0, new_store = 0;
  // The metric sums run on a second stream of the library, from the moment the ingest's
  // slot ids are complete: they overlap the host's reading of the counters, the publish
  // and the ordering.  Per-workgroup LDS maps, flushed through staging buckets of slots;
  // two workgroups per CU (run one after the other) halve the distinct slots each map
  // must hold, so fewer events overflow into device atomics.  (A test setting keeps
  // everything on the caller's stream, the path taken when no second stream can be
  // created.)
  SideGuard side_guard;
  Event slots_ready;
  AggStage stg{};
  const int agg_grid = (int)std::max<int64_t>(1, std::min<int64_t>((N + 8191) / 8192, (int64_t)cu_count() * 2));
  if (N > 0) {
    hipStream_t ss = env_int("CCT_TEST_ONE_STREAM", 0) ? nullptr : side_guard.acquire();
    if (ss) side = ss;
    if (side != s && !slots_ready.ev) return fail(CCT_EDEVICE, "event creation failed");
  }
  if (N > 0) {
    if (!slot_of.alloc((size_t)N * 4)) return fail(CCT_ENOMEM, "device allocation failed");
    for (int attempt = 0;; ++attempt) {
      if (attempt > 12) return fail(CCT_EOVERFLOW, "unique-path table cannot grow further");
      const int64_t max_new = (int64_t)std::min<uint64_t>(t->cap, (uint64_t)N);  // distinct paths of the batch
      if (!delta.alloc(t->cap * m * 8) || !new_slots.alloc(t->cap * 4) ||
          !cpart.alloc((size_t)collect_blocks(t->cap) * 16) || !nsrc.alloc((size_t)max_new * 16) ||
          !nlen.alloc((size_t)(max_new + 1) * 8))
        return fail(CCT_ENOMEM, "device allocation failed");
      AGG_TRY(hipMemsetAsync(delta.p, 0, t->cap * m * 8, s));
      AGG_TRY(hipMemsetAsync(dctr, 0, kCtrCount * 8, s));
      IngestArgs a{};
      a.off = p->offsets; a.fr = p->frames;
      a.n_events = N; a.n_frames = p->n_frames;
      a.slot = t->slot.as<Slot>(); a.cap_mask = t->cap - 1; a.hash_mask = hash_mask;
      a.slot_of = slot_of.as<uint32_t>();
      a.pframes = t->pframes.as<uint32_t>(); a.pstart = t->pstart.as<int64_t>(); a.plen = t->plen.as<uint32_t>();
      a.ctr = dctr;
      // one workgroup per CU; every wave owns an equal share of the events
      const int64_t wg_needed = (N + kIngestThreads / 64 - 1) / (kIngestThreads / 64);
      const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(wg_needed, (int64_t)cu_count()));
      tm.mark(1, s);
      launch_ingest(a, grid, s);
      tm.mark(2, s);
      launch_collect_new(t->slot.as<Slot>(), t->cap, p->offsets, new_slots.as<uint32_t>(), nsrc.as<int64_t>(),
                         nlen.as<uint64_t>(), dctr, cpart.as<unsigned long long>(), s);
      claimed = true;  // (from the launch on: the table may hold this call's claims)
      AGG_TRY(hipGetLastError());
      {
        // (the side stream's work, the staging's zeroing included, starts after the collection)
        if (side != s) {
          AGG_TRY(hipEventRecord(slots_ready.ev, s));
          AGG_TRY(hipStreamWaitEvent(side, slots_ready.ev, 0));
        }
        cct_status sst = setup_stage(m, t->cap, agg_grid, agg_count, agg_keys, agg_sums, stg, side);
        if (sst) return undo(sst);
        launch_aggregate(slot_of.as<uint32_t>(), p->metrics, N, m, delta.as<uint64_t>(), t->cap, agg_grid, stg, side);
        AGG_TRY(hipGetLastError());
      }
      AGG_TRY(hipMemcpyAsync(hs, dctr, kCtrCount * 8, hipMemcpyDeviceToHost, s));
      AGG_TRY(spin_sync(s));
      if (hs[kCtrError]) return undo(fail(CCT_EINVAL, "malformed offsets"));
      if (hs[kCtrOverflow]) {
        // the sums of this attempt are discarded: their buffers are reused once idle
        if (side != s) AGG_TRY(hipStreamSynchronize(side));
        // a larger table holding only the tree's paths; the old one, with this call's
        // claims, is discarded once rehash has synchronised the stream
        cct_status st = rehash(t, t->cap * 4, hash_mask, s);
        if (st) return undo(st);
        claimed = false;
        continue;
      }
      n_new = hs[kCtrNew];
      claimed = n_new > 0;
      new_frames = hs[kCtrNewLen];
      new_store = hs[kCtrNewFrames];
      break;
    }
  }

  // ---- allocate everything the rest of the call needs (rollback possible until here)
  const int64_t D = t->d + (int64_t)n_new;
  const int64_t sum_len = t->sum_len + (int64_t)new_frames;
  if (sum_len + 1 > (int64_t)0xFFFFFFFE) return undo(fail(CCT_EOVERFLOW, "tree would exceed 2^32-2 nodes"));
  // this batch's statistics, staged in path-range buckets when there are few enough of them
  // (a test setting forces device atomics instead); allocated before anything of the tree
  // changes
  Buf sg_pos, sg_ev_path, sg_ev_w, sg_map_key, sg_map_rec, sg_hist, sg_off, sg_blk, sg_wg, sg_st_path, sg_st_w,
      sg_st_key, sg_st_rec;
  StatStage sst{};
  const bool keep_stats = t->stats && N > 0;
  const int st_grid = (int)std::max<int64_t>(1, std::min<int64_t>((N + 8191) / 8192, (int64_t)cu_count() * 2));
  if (keep_stats) {
    if (!sg_pos.alloc(t->cap * 4)) return undo(fail(CCT_ENOMEM, "device allocation failed"));
    // buckets of 2^bshift paths: about 256 of them, each within the reduction's LDS
    const int64_t D_all = t->d + (int64_t)n_new;
    int bshift = 6;
    while (bshift < stats_bucket_shift(m) && (D_all >> bshift) > 256) ++bshift;
    const int64_t nbk = (D_all + (1ll << bshift) - 1) >> bshift;
    if (nbk <= stats_max_buckets() && !env_int("CCT_TEST_STATS_ATOMIC", 0)) {
      const int64_t me = stats_staged_entries(m), R = 1 + 3 * (int64_t)m, rows = nbk * st_grid;
      const int64_t nmap = st_grid * me;
      if (!sg_ev_path.alloc(N * 4) || !sg_ev_w.alloc(N * m * 8) || !sg_map_key.alloc(nmap * 4) ||
          !sg_map_rec.alloc(nmap * R * 8) || !sg_hist.alloc(2 * rows * 8) || !sg_off.alloc(2 * (rows + 1) * 8) ||
          !sg_blk.alloc((rows / 1024 + 2) * 8) || !sg_wg.alloc(st_grid * 8) || !sg_st_path.alloc(N * 4) ||
          !sg_st_w.alloc(N * m * 8) || !sg_st_key.alloc(nmap * 4) || !sg_st_rec.alloc(nmap * R * 8))
        return undo(fail(CCT_ENOMEM, "device allocation failed"));
      sst.bshift = bshift; sst.nbuckets = nbk; sst.grid = st_grid; sst.map_entries = me;
      sst.ev_path = sg_ev_path.as<uint32_t>(); sst.ev_w = sg_ev_w.as<uint64_t>();
      sst.map_key = sg_map_key.as<uint32_t>(); sst.map_rec = sg_map_rec.as<uint64_t>();
      sst.hist_ev = sg_hist.as<uint64_t>(); sst.hist_map = sst.hist_ev + rows;
      sst.off_ev = sg_off.as<uint64_t>(); sst.off_map = sst.off_ev + rows + 1;
      sst.wg_count = sg_wg.as<uint32_t>();
      sst.st_ev_path = sg_st_path.as<uint32_t>(); sst.st_ev_w = sg_st_w.as<uint64_t>();
      sst.st_map_key = sg_st_key.as<uint32_t>(); sst.st_map_rec = sg_st_rec.as<uint64_t>();
    }
  }
  const int64_t store_need = t->store_used + (int64_t)new_store;
  const int64_t dneed = std::max<int64_t>(D, 1);
  cct_tree old_arrays_holder;  // receives replaced buffers, released on return
  {
    cct_status st = CCT_OK;
    if (store_need > t->store_cap || !t->pframes.p) {
      const int64_t ncap = std::max<int64_t>(store_need + store_need / 2, 1024);
      Buf f2, c2;
      if (!f2.alloc(ncap * 4) || !c2.alloc((ncap / kStoreAlign + 1) * 8)) return undo(fail(CCT_ENOMEM, "device allocation failed"));
      if (t->store_used) {
        if (hipMemcpyAsync(f2.p, t->pframes.p, t->store_used * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(c2.p, t->pcp.p, (t->store_used / kStoreAlign) * 8, hipMemcpyDeviceToDevice, s) != hipSuccess)
          return undo(fail(CCT_EDEVICE, "copy failed"));
      }
      old_arrays_holder.pframes = std::move(t->pframes);
      old_arrays_holder.pcp = std::move(t->pcp);
      t->pframes = std::move(f2);
      t->pcp = std::move(c2);
      t->store_cap = ncap;
    }
    if (dneed > t->dcap || !t->pstart.p) {
      const int64_t ncap = std::max<int64_t>(dneed + dneed / 2, 256);
      Buf a1, a2, a3;
      if (!a1.alloc(ncap * 8) || !a2.alloc(ncap * 4) || !a3.alloc(ncap * 4))
        return undo(fail(CCT_ENOMEM, "device allocation failed"));
      if (t->d) {
        if (hipMemcpyAsync(a1.p, t->pstart.p, t->d * 8, hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(a2.p, t->plen.p, t->d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
            hipMemcpyAsync(a3.p, t->pslot.p, t->d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
          return undo(fail(CCT_EDEVICE, "copy failed"));
      }
      old_arrays_holder.pstart = std::move(t->pstart);
      old_arrays_holder.plen = std::move(t->plen);
      old_arrays_holder.pslot = std::move(t->pslot);
      t->pstart = std::move(a1); t->plen = std::move(a2); t->pslot = std::move(a3);
      t->dcap = ncap;
    }
    (void)st;
  }
  // the paths' sums (and statistics) after this batch, in fresh arrays: the tree's own
  // stay as they are until the commit
  Buf nsums, ncnt, nmin, nsq;
  if (!nsums.alloc(t->dcap * m * 8)) return undo(fail(CCT_ENOMEM, "device allocation failed"));
  if (t->stats) {
    if (!ncnt.alloc(t->dcap * 8) || !nmin.alloc(t->dcap * m * 8) || !nsq.alloc(t->dcap * m * 16))
      return undo(fail(CCT_ENOMEM, "device allocation failed"));
    if (t->d &&
        (hipMemcpyAsync(ncnt.p, t->pcnt.p, t->d * 8, hipMemcpyDeviceToDevice, s) != hipSuccess ||
         hipMemcpyAsync(nmin.p, t->pmin.p, t->d * m * 8, hipMemcpyDeviceToDevice, s) != hipSuccess ||
         hipMemcpyAsync(nsq.p, t->psq.p, t->d * m * 16, hipMemcpyDeviceToDevice, s) != hipSuccess))
      return undo(fail(CCT_EDEVICE, "copy failed"));
  }
  const int C = 1 + m;
  const int64_t n1 = D + 1;
  const int levels = floor_log2((uint64_t)n1) + 1;
  const int64_t nblk = (D + 1023) / 1024 + 1;
  const int64_t u_max = sum_len + 1;
  Buf order, order_tmp, lcp, scan_in, scan_out, scan_blk, sparse, chain, win_path, cursor, nstart, nblkbuf;
  Buf n_parent, n_frame, n_depth, n_subend, n_excl, n_incl;  // canonical arrays of the new tree
  if (!order.alloc(dneed * 4) || !order_tmp.alloc(dneed * 4) || !lcp.alloc(n1 * 4) || !scan_in.alloc(dneed * C * 8) ||
      !scan_out.alloc(n1 * C * 8) || !scan_blk.alloc(nblk * C * 8) || !sparse.alloc((int64_t)levels * n1 * 4) ||
      !chain.alloc(dneed * 4) || !win_path.alloc((u_max / 64 + 2) * 4) || !cursor.alloc(64) || !n_parent.alloc(u_max * 4) || !n_subend.alloc(u_max * 4) ||
      !n_frame.alloc(u_max * 4) || !n_depth.alloc(u_max * 4) || !n_excl.alloc(u_max * m * 8) ||
      !n_incl.alloc(u_max * m * 8) || !nstart.alloc((n_new + 1) * 8) ||
      !nblkbuf.alloc(((int64_t)n_new / 1024 + 2) * 8))
    return undo(fail(CCT_ENOMEM, "device allocation failed"));

  // sorting scratch, allocated before the tree is touched
  const bool exact_sort = env_int("CCT_TEST_EXACT_SORT", 0) != 0;
  // Pass 0 ranks the paths through the block trie (trie.hip); if that is not usable (a
  // hash collision, an oversized sibling group) or its order fails the exact check,
  // pass 1 sorts by exact comparisons.  A test setting forces the comparison sort.
  const int64_t nblocks = store_need / kStoreAlign;
  // a merge keeps the previous order: only this call's new paths are sorted, then
  // merged in (a test setting forces the full sort)
  const bool incremental = t->d > 0 && t->order.p && !exact_sort && !env_int("CCT_TEST_FULL_SORT", 0);
  const bool use_trie = !incremental && !exact_sort && !env_int("CCT_TEST_MERGE_SORT", 0) && D > 0;
  Buf merge_scratch;
  if (incremental && !merge_scratch.alloc(std::max<int64_t>(2 * (int64_t)n_new, 1) * 4))
    return undo(fail(CCT_ENOMEM, "device allocation failed"));
  Buf tr_key, tr_info, tr_bpos, tr_occ, tr_par, tr_cnt, tr_end, tr_hist, tr_gstart, tr_cidx, tr_rb, tr_lg, tr_spl, tr_bc, tr_grp, tr_grp2, tr_pos,
      tr_c, tr_cs, tr_blk, tr_lists, tr_ctr;
  TrieArgs ta{};
  if (use_trie) {
    const uint64_t tcap = pow2_at_least(std::max<uint64_t>(2 * (uint64_t)nblocks, 1024));
    const int64_t nbk = std::max<int64_t>(nblocks, 1);
    const int64_t list_cap = nbk + 1024;
    const int64_t large_cap = nbk / 512 + 1;  // groups of more than 512 siblings (split into buckets)
    const int64_t scan_rows = std::max<int64_t>((int64_t)tcap + 1, nbk);
    if (!tr_key.alloc(tcap * 8) || !tr_info.alloc(tcap * 8) || !tr_bpos.alloc(nbk * 8) || !tr_occ.alloc(nbk * 4) ||
        !tr_par.alloc(tcap * 4) || !tr_cnt.alloc(tcap * 4) || !tr_end.alloc((tcap + 1) * 4) ||
        !tr_hist.alloc((tcap + 1) * 8) || !tr_gstart.alloc((tcap + 2) * 8) || !tr_cidx.alloc(tcap * 4) ||
        !tr_rb.alloc(1024 * 4) || !tr_lg.alloc((tcap + 1) * 4) || !tr_spl.alloc(large_cap * 256 * 4) ||
        !tr_bc.alloc(large_cap * 256 * 4) ||
        !tr_grp.alloc(nbk * 4) || !tr_grp2.alloc(nbk * 4) || !tr_pos.alloc(tcap * 4) || !tr_c.alloc(nbk * 8) ||
        !tr_cs.alloc((nbk + 1) * 8) || !tr_blk.alloc((scan_rows / 1024 + 2) * 8) || !tr_lists.alloc(4 * list_cap * 8) ||
        !tr_ctr.alloc(64))
      return undo(fail(CCT_ENOMEM, "device allocation failed"));
    ta.d = D; ta.nblocks = nblocks; ta.cap = tcap;
    ta.pframes = t->pframes.as<uint32_t>(); ta.pcp = t->pcp.as<uint64_t>(); ta.pstart = t->pstart.as<int64_t>();
    ta.plen = t->plen.as<uint32_t>();
    ta.tkey = tr_key.as<uint64_t>(); ta.tinfo = tr_info.as<uint64_t>(); ta.bpos = tr_bpos.as<uint64_t>();
    ta.occ = tr_occ.as<uint32_t>(); ta.nparent = tr_par.as<uint32_t>(); ta.ncount = tr_cnt.as<uint32_t>();
    ta.nend = tr_end.as<uint32_t>(); ta.hist = tr_hist.as<uint64_t>(); ta.gstart = tr_gstart.as<uint64_t>();
    ta.cidx = tr_cidx.as<uint32_t>(); ta.rootbase = tr_rb.as<uint32_t>(); ta.grouped = tr_grp.as<uint32_t>(); ta.grouped2 = tr_grp2.as<uint32_t>();
    ta.posof = tr_pos.as<uint32_t>(); ta.cnt = tr_c.as<uint64_t>(); ta.cnt_scan = tr_cs.as<uint64_t>();
    ta.scan_blk = tr_blk.as<uint64_t>(); ta.lists = tr_lists.as<uint64_t>(); ta.list_cap = list_cap; ta.large_cap = large_cap;
    ta.lgroup = tr_lg.as<uint32_t>(); ta.spl = tr_spl.as<uint32_t>(); ta.bcnt = tr_bc.as<uint32_t>();
    ta.ctr = tr_ctr.as<unsigned long long>(); ta.order = order.as<uint32_t>();
  }

  Timer ts;
  g_stats_ms = 0;

  // ---- publish new paths, fold this call's sums into the old ones -----------------------
  // events that order the side stream's fold after the publish, and the emission after
  // the fold: created before anything is published
  Event published_ev, folded, trie_fork, trie_mid, trie_join;
  if (N > 0 && side != s && (!published_ev.ev || !folded.ev)) return undo(fail(CCT_EDEVICE, "event creation failed"));
  AGG_TRY(hipMemsetAsync(cursor.p, 0, 64, s));
  if (n_new) {
    // place the new paths in the store: exclusive scan of their padded lengths (listed
    // by collect_new with their first frames and lengths)
    launch_scan(nlen.as<uint64_t>(), (int64_t)n_new, 1, nblkbuf.as<uint64_t>(), nstart.as<uint64_t>(), s);
    AGG_TRY(hipMemcpyAsync(cursor.p, nstart.as<uint64_t>() + n_new, 8, hipMemcpyDeviceToDevice, s));
    PublishArgs pa{};
    pa.off = p->offsets; pa.fr = p->frames; pa.n_frames = p->n_frames; pa.slot = t->slot.as<Slot>();
    pa.new_slots = new_slots.as<uint32_t>(); pa.n_new = (int64_t)n_new; pa.d_old = t->d;
    pa.pframes = t->pframes.as<uint32_t>(); pa.pcp = t->pcp.as<uint64_t>();
    pa.pstart = t->pstart.as<int64_t>(); pa.plen = t->plen.as<uint32_t>(); pa.pslot = t->pslot.as<uint32_t>();
    pa.store_used = t->store_used; pa.starts = nstart.as<uint64_t>();
    pa.src_len = nsrc.as<int64_t>();
    // a test setting keeps fewer bits of the checkpoint hashes, so that the fast orders
    // meet colliding prefixes and the exact comparison sort has to take over
    const int cp_bits = (int)env_int("CCT_TEST_CP_HASH_BITS", 64);
    pa.cp_mask = cp_bits >= 64 ? ~0ull : ((1ull << (cp_bits < 1 ? 1 : cp_bits)) - 1);
    published = true;  // from here on, a failure empties the published slots
    launch_publish(pa, s);
  }
  // every path's sums, once both the side stream's aggregation and the publish (which
  // records the new paths' slots) are done; the emission waits for them
  if (N > 0) {
    if (side != s) {
      AGG_TRY(hipEventRecord(published_ev.ev, s));
      AGG_TRY(hipStreamWaitEvent(side, published_ev.ev, 0));
    }
    launch_fold_sums(D, t->d, m, t->pslot.as<uint32_t>(), delta.as<uint64_t>(), t->psums.as<uint64_t>(),
                     nsums.as<uint64_t>(), side);
    if (side != s) AGG_TRY(hipEventRecord(folded.ev, side));
  }
  if (keep_stats) {  // the batch's samples into the fresh path arrays (new paths start empty)
    ts.mark(0, s);
    PathStats ps{ncnt.as<uint64_t>(), nmin.as<uint64_t>(), nsq.as<uint64_t>()};
    launch_stats_prepare(D, t->d, m, t->pslot.as<uint32_t>(), sg_pos.as<uint32_t>(), ps, s);
    launch_stats_agg(slot_of.as<uint32_t>(), sg_pos.as<uint32_t>(), p->metrics, N, m, D, st_grid, ps, sst,
                     sg_blk.as<uint64_t>(), s);
    ts.mark(1, s);
  }
  AGG_TRY(hipGetLastError());
  tm.mark(3, s);
  // test setting: fail once everything is published and folded, to check that the
  // tree is left as it was
  if (env_int("CCT_TEST_FAIL_AFTER_PUBLISH", 0)) return undo(fail(CCT_EDEVICE, "test failure after publish"));

  // ---- A5-A9: canonical order and node arrays ------------------------------------------
  CanonArgs ca{};
  ca.d = D; ca.m = m; ca.exact = exact_sort ? 1 : 0;
  ca.pframes = t->pframes.as<uint32_t>(); ca.pcp = t->pcp.as<uint64_t>(); ca.pstart = t->pstart.as<int64_t>();
  ca.plen = t->plen.as<uint32_t>(); ca.psums = nsums.as<uint64_t>();
  ca.order = order.as<uint32_t>(); ca.order_tmp = order_tmp.as<uint32_t>(); ca.lcp = lcp.as<uint32_t>();
  ca.scan_in = scan_in.as<uint64_t>(); ca.scan_out = scan_out.as<uint64_t>(); ca.scan_blk = scan_blk.as<uint64_t>();
  ca.scan_blocks = nblk; ca.sparse = sparse.as<uint32_t>(); ca.levels = levels;
  ca.chain_parent = chain.as<uint32_t>(); ca.win_path = win_path.as<uint32_t>(); ca.u_max = u_max;
  ca.parent = n_parent.as<uint32_t>(); ca.frame = n_frame.as<uint32_t>(); ca.depth = n_depth.as<uint32_t>();
  ca.subend = n_subend.as<uint32_t>();
  ca.excl = n_excl.as<uint64_t>(); ca.incl = n_incl.as<uint64_t>();
  ca.u_out = cursor.as<unsigned long long>() + 2;
  ca.grid_nodes = (int)std::max<int64_t>(1, std::min<int64_t>((u_max + 255) / 256, (int64_t)cu_count() * 16));
  // 0: block trie, 1: comparison sort with checkpoint hashes, 2: exact comparisons only,
  // 3: the previous order with this call's new paths merged in
  for (int mode = incremental ? 3 : (use_trie ? 0 : (ca.exact ? 2 : 1));;) {
    CanonArgs run = ca;
    run.exact = mode == 2 ? 1 : 0;
    if (mode == 0) launch_trie_sort(ta, s, side, trie_fork.ev, trie_mid.ev, trie_join.ev);
    else if (mode == 3) launch_merge_order(run, t->order.as<uint32_t>(), t->d, merge_scratch.as<uint32_t>(), s);
    else launch_sort(run, s);
    tm.mark(4, s);
    if (N > 0 && side != s) AGG_TRY(hipStreamWaitEvent(s, folded.ev, 0));  // the emission reads the sums
    launch_canon(run, s);
    AGG_TRY(hipGetLastError());
    tm.mark(5, s);
    AGG_TRY(hipMemcpyAsync(hs, cursor.p, 64, hipMemcpyDeviceToHost, s));
    if (mode == 0) AGG_TRY(hipMemcpyAsync(hs + 8, ta.ctr, 64, hipMemcpyDeviceToHost, s));
    AGG_TRY(spin_sync(s));
    const bool trie_failed = mode == 0 && hs[8 + kTrieCtrFail] != 0;
    if (!hs[3] && !trie_failed) {  // order verified strictly increasing
      if (run.order != ca.order) std::swap(order, order_tmp);
      break;
    }
    if (mode == 2) return undo(fail(CCT_EDEVICE, "canonical order failed exact verification"));
    if (mode == 0 && env_int("CCT_TEST_REQUIRE_TRIE", 0)) return undo(fail(CCT_EDEVICE, "block-trie order not usable"));
    mode = 2;  // a hash collision misled the fast order: sort again with exact compares
    AGG_TRY(hipMemsetAsync(cursor.as<unsigned long long>() + 2, 0, 16, s));
  }
  tm.collect(N > 0);
  if (keep_stats && ts.ok) g_stats_ms = ts.span(0, 1);

  // ---- commit -------------------------------------------------------------------------------
  t->store_used += (int64_t)hs[0];
  t->d = D;
  t->sum_len = sum_len;
  t->u = (int64_t)hs[2];
  t->parent = std::move(n_parent); t->frame = std::move(n_frame); t->depth = std::move(n_depth);
  t->subend = std::move(n_subend);
  t->bu_k = -1;        // the bottom-up view of the old tree is stale
  t->q_ready = false;  // and so is the query index
  t->excl = std::move(n_excl); t->incl = std::move(n_incl);
  t->order = std::move(order); t->lcp = std::move(lcp); t->scan_out = std::move(scan_out);
  t->psums = std::move(nsums);
  if (t->stats) { t->pcnt = std::move(ncnt); t->pmin = std::move(nmin); t->psq = std::move(nsq); }
  return CCT_OK;
#undef AGG_TRY
}

}  // namespace

extern "C" {

cct_status build_tree(const cct_paths *events, void *hip_stream, bool stats, cct_tree **out) {
  AllocHook hook;
  g_join_ms = 0;
  clear_error();
  if (!out) return fail(CCT_EINVAL, "out is NULL");
  cct_status st = check_paths(events, true);
  if (st) return st;
  hipStream_t s = (hipStream_t)hip_stream;
  cct_tree *t = new (std::nothrow) cct_tree;
  if (!t) return fail(CCT_ENOMEM, "host allocation failed");
  (void)hipGetDevice(&t->device);
  t->m = events->n_metrics;
  t->stats = stats;
  const int64_t N = events->n_events;
  int64_t cap = env_int("CCT_TEST_TABLE_CAP", 0);
  if (cap <= 0) cap = (int64_t)std::min<uint64_t>(pow2_at_least((uint64_t)std::max<int64_t>(2 * N, 1024)), 1ull << 21);
  cap = (int64_t)pow2_at_least((uint64_t)std::max<int64_t>(cap, 16));
  if (!t->slot.alloc(cap * sizeof(Slot))) { delete t; return fail(CCT_ENOMEM, "device allocation failed"); }
  t->cap = (uint64_t)cap;
  if (hipMemsetAsync(t->slot.p, 0xFF, cap * sizeof(Slot), s) != hipSuccess) {
    (void)hipGetLastError();
    delete t;
    return fail(CCT_EDEVICE, "memset failed");
  }
  st = aggregate(t, events, s);
  if (st) { delete t; return st; }
  *out = t;
  return CCT_OK;
}

cct_status cct_build(const cct_paths *events, void *hip_stream, cct_tree **out) {
  return build_tree(events, hip_stream, false, out);
}

cct_status cct_build_stats(const cct_paths *events, void *hip_stream, cct_tree **out) {
  return build_tree(events, hip_stream, true, out);
}

cct_status cct_merge(cct_tree *tree, const cct_paths *chunk, void *hip_stream) {
  AllocHook hook;
  clear_error();
  g_join_ms = 0;
  if (!tree) return fail(CCT_EINVAL, "tree is NULL");
  cct_status st = check_paths(chunk, true);
  if (st) return st;
  if (chunk->n_metrics != tree->m) return fail(CCT_EMISMATCH, "metric count differs from the tree's");
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  return aggregate(tree, chunk, (hipStream_t)hip_stream);
}

cct_status cct_merge_activity(cct_tree *tree, const cct_paths *registry, const uint64_t *reg_corr_ids,
                              const cct_activity *act, void *hip_stream, int64_t *n_unmatched) {
  AllocHook hook;  // counts the join's and the merge's allocations together
  clear_error();
  g_join_ms = 0;
  if (!tree || !registry || !act) return fail(CCT_EINVAL, "NULL argument");
  const int64_t G = registry->n_events, R = act->n_records;
  if (G < 0 || registry->n_frames < 0 || R < 0) return fail(CCT_EINVAL, "negative size");
  if (G > CCT_MAX_EVENTS || R > CCT_MAX_EVENTS) return fail(CCT_EOVERFLOW, "too many paths or records in one call");
  if (!registry->offsets || (registry->n_frames > 0 && !registry->frames) || (G > 0 && !reg_corr_ids))
    return fail(CCT_EINVAL, "registry pointer is NULL");
  if (act->n_metrics < 1 || act->n_metrics > CCT_MAX_METRICS) return fail(CCT_EINVAL, "n_metrics out of range");
  if (R > 0 && (!act->corr_ids || !act->metrics)) return fail(CCT_EINVAL, "activity pointer is NULL");
  if (((uintptr_t)registry->offsets & 7) || ((uintptr_t)registry->frames & 3) || ((uintptr_t)reg_corr_ids & 7) ||
      ((uintptr_t)act->corr_ids & 7) || ((uintptr_t)act->metrics & 7))
    return fail(CCT_EINVAL, "misaligned pointer");
  if (act->n_metrics != tree->m) return fail(CCT_EMISMATCH, "metric count differs from the tree's");
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  hipStream_t s = (hipStream_t)hip_stream;
  const int32_t m = tree->m;
  unsigned long long *hs = host_scratch();
  if (!hs) return fail(CCT_ENOMEM, "pinned host allocation failed");
  if (G == 0 || R == 0) {  // nothing can match: no device work
    if (n_unmatched) *n_unmatched = R;
    return CCT_OK;
  }
  Timer tm;
  tm.mark(0, s);
  // ---- table of registered IDs, the join, per-path sums -------------------------------
  Buf table, rec_reg, ref, sums, ctr, rows, scan, scan_blk, add_list, add_cnt;
  ActivityArgs a{};
  a.n_reg = G; a.reg_n_frames = registry->n_frames; a.reg_off = registry->offsets; a.reg_corr = reg_corr_ids;
  a.n_rec = R; a.rec_corr = act->corr_ids;
  // the range of the registered IDs decides between the direct and the hash table
  if (!ctr.alloc(kActCtrCount * 8)) return fail(CCT_ENOMEM, "device allocation failed");
  a.ctr = ctr.as<unsigned long long>();
  HIP_TRY(hipMemsetAsync(ctr.p, 0, kActCtrCount * 8, s));
  HIP_TRY(hipMemsetAsync(a.ctr + kActCtrMin, 0xFF, 8, s));
  launch_corr_range(a, s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(hs, a.ctr + kActCtrMin, 16, hipMemcpyDeviceToHost, s));
  HIP_TRY(spin_sync(s));
  a.id_min = hs[0];
  a.id_span = hs[1] - hs[0];
  a.dense = a.id_span < 4 * (uint64_t)G;
  const uint64_t cap = a.dense ? a.id_span + 1 : pow2_at_least((uint64_t)std::max<int64_t>(2 * G, 64));
  const size_t table_bytes = a.dense ? cap * 4 : cap * sizeof(CorrSlot);
  if (!table.alloc(table_bytes) || !rec_reg.alloc((size_t)R * 4) || !ref.alloc((size_t)G * 4) ||
      !sums.alloc((size_t)G * m * 8) || !rows.alloc((size_t)G * 16) ||
      !scan.alloc(((size_t)G + 1) * 16) || !scan_blk.alloc(((size_t)G / 1024 + 2) * 16) ||
      !add_list.alloc(((size_t)R + (size_t)corr_sums_grid(R) * 256) * 4) || !add_cnt.alloc((size_t)corr_sums_grid(R) * 4))
    return fail(CCT_ENOMEM, "device allocation failed");
  HIP_TRY(hipMemsetAsync(table.p, 0, table_bytes, s));
  HIP_TRY(hipMemsetAsync(ref.p, 0, (size_t)G * 4, s));
  if (a.dense) a.dtab = table.as<uint32_t>();
  else { a.table = table.as<CorrSlot>(); a.cap_mask = cap - 1; }
  a.rec_reg = rec_reg.as<uint32_t>(); a.ref = ref.as<uint32_t>();
  launch_corr_table(a, s);
  launch_corr_join(a, s);
  launch_corr_sums(a, act->metrics, m, sums.as<uint64_t>(), add_list.as<uint32_t>(), add_cnt.as<uint32_t>(), s);
  launch_compact_lengths(a, rows.as<uint64_t>(), s);
  launch_scan(rows.as<uint64_t>(), G, 2, scan_blk.as<uint64_t>(), scan.as<uint64_t>(), s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(hs, ctr.p, 2 * 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipMemcpyAsync(hs + 2, scan.as<uint64_t>() + 2 * G, 16, hipMemcpyDeviceToHost, s));
  HIP_TRY(spin_sync(s));
  const unsigned long long err = hs[kActCtrError], unmatched = hs[kActCtrUnmatched];
  const int64_t n_used = (int64_t)hs[2], n_fr = (int64_t)hs[3];
  if (err & kActBadOffsets) return fail(CCT_EINVAL, "malformed registry offsets");
  if (err & kActRepeatedId) return fail(CCT_EINVAL, "a correlation ID is registered twice");
  if (err) return fail(CCT_EDEVICE, "correlation-ID table overflow");
  // ---- the batch of referenced paths with their summed metrics, merged ---------------
  // (every registered path referenced: the registry is the batch, nothing is copied)
  cct_paths batch{};
  batch.n_events = n_used; batch.n_frames = n_fr; batch.n_metrics = m;
  Buf b_off, b_src, b_fr, b_met;
  if (n_used == G) {
    batch.offsets = registry->offsets; batch.frames = registry->frames; batch.metrics = sums.as<uint64_t>();
  } else {
    if (!b_off.alloc(((size_t)n_used + 1) * 8) || !b_src.alloc(((size_t)n_used + 1) * 8) ||
        !b_fr.alloc((size_t)n_fr * 4) || !b_met.alloc((size_t)n_used * m * 8))
      return fail(CCT_ENOMEM, "device allocation failed");
    launch_compact_gather(a, registry->frames, scan.as<uint64_t>(), sums.as<uint64_t>(), m, n_used, n_fr,
                          b_off.as<int64_t>(), b_src.as<int64_t>(), b_fr.as<uint32_t>(), b_met.as<uint64_t>(), s);
    batch.offsets = b_off.as<int64_t>(); batch.frames = b_fr.as<uint32_t>(); batch.metrics = b_met.as<uint64_t>();
  }
  HIP_TRY(hipGetLastError());
  tm.mark(1, s);
  HIP_TRY(spin_sync(s));
  const double join_ms = tm.ok ? tm.span(0, 1) : 0.0;
  cct_status st = aggregate(tree, &batch, s);
  if (st) return st;
  g_join_ms = join_ms;
  if (n_unmatched) *n_unmatched = (int64_t)unmatched;
  return CCT_OK;
}

namespace {

// The bottom-up view of `t` into t->bu_* (see bottomup.hip).  Nothing of the tree changes
// on failure.
cct_status compute_bottom_up(cct_tree *t, hipStream_t s) {
  const int64_t n = t->u - 1;  // nodes other than the root
  const int64_t U = t->u;
  const int32_t m = t->m;
  unsigned long long *hs = host_scratch();
  if (!hs) return fail(CCT_ENOMEM, "pinned host allocation failed");
  if (n <= 0) {
    t->bu_k = 0;
    return CCT_OK;
  }
  const int64_t rb = radix_blocks(n), hist_rows = 256 * rb;
  const int64_t scan_rows = std::max<int64_t>(hist_rows, n);
  Buf keys, vals, keys_t, vals_t, hist, offs, scan_blk, head, gscan, tag, mx, ms_blk, gstart, slot_ex, slot_in;
  if (!keys.alloc(n * 4) || !vals.alloc(n * 4) || !keys_t.alloc(n * 4) || !vals_t.alloc(n * 4) ||
      !hist.alloc(hist_rows * 8) || !offs.alloc((hist_rows + 1) * 8) || !scan_blk.alloc((scan_rows / 1024 + 2) * 8) ||
      !head.alloc(n * 8) || !gscan.alloc((n + 1) * 8) || !tag.alloc(n * 8) || !mx.alloc(n * 8) ||
      !ms_blk.alloc((maxscan_blocks(n) + 1) * 8) || !gstart.alloc((n + 1) * 8) || !slot_ex.alloc(U * 4) ||
      !slot_in.alloc(U * 4))
    return fail(CCT_ENOMEM, "device allocation failed");
  Timer tm;
  tm.mark(0, s);
  uint32_t *K = keys.as<uint32_t>(), *V = vals.as<uint32_t>();
  launch_bu_keys(t->frame.as<uint32_t>(), n, K, V, s);
  launch_radix_sort(K, V, keys_t.as<uint32_t>(), vals_t.as<uint32_t>(), n, hist.as<uint64_t>(), offs.as<uint64_t>(),
                    scan_blk.as<uint64_t>(), s);
  launch_bu_heads(K, n, head.as<uint64_t>(), s);
  launch_scan(head.as<uint64_t>(), n, 1, scan_blk.as<uint64_t>(), gscan.as<uint64_t>(), s);
  launch_bu_tag(V, head.as<uint64_t>(), gscan.as<uint64_t>(), t->subend.as<uint32_t>(), n, tag.as<uint64_t>(),
                gstart.as<int64_t>(), s);
  launch_maxscan(tag.as<uint64_t>(), n, ms_blk.as<uint64_t>(), mx.as<uint64_t>(), s);
  launch_bu_slots(V, head.as<uint64_t>(), gscan.as<uint64_t>(), mx.as<uint64_t>(), n, slot_ex.as<uint32_t>(),
                  slot_in.as<uint32_t>(), s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(hs, gscan.as<uint64_t>() + n, 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(spin_sync(s));
  const int64_t G = (int64_t)hs[0];
  // per-group sums: exclusive sums of every node, inclusive sums of the topmost ones
  Buf f_out, e_out, i_out, cnt_e, keys_e, sums_e, cnt_i, keys_i, sums_i;
  const int agg_grid = (int)std::max<int64_t>(1, std::min<int64_t>((U + 8191) / 8192, (int64_t)cu_count() * 2));
  AggStage st_e{}, st_i{};
  if (!f_out.alloc(G * 4) || !e_out.alloc(G * m * 8) || !i_out.alloc(G * m * 8))
    return fail(CCT_ENOMEM, "device allocation failed");
  cct_status st = setup_stage(m, (uint64_t)G, agg_grid, cnt_e, keys_e, sums_e, st_e, s);
  if (!st) st = setup_stage(m, (uint64_t)G, agg_grid, cnt_i, keys_i, sums_i, st_i, s);
  if (st) return st;
  HIP_TRY(hipMemsetAsync(e_out.p, 0, G * m * 8, s));
  HIP_TRY(hipMemsetAsync(i_out.p, 0, G * m * 8, s));
  launch_bu_frames(K, gstart.as<int64_t>(), G, f_out.as<uint32_t>(), s);
  launch_aggregate(slot_ex.as<uint32_t>(), t->excl.as<uint64_t>(), U, m, e_out.as<uint64_t>(), (uint64_t)G, agg_grid,
                   st_e, s);
  launch_aggregate(slot_in.as<uint32_t>(), t->incl.as<uint64_t>(), U, m, i_out.as<uint64_t>(), (uint64_t)G, agg_grid,
                   st_i, s);
  HIP_TRY(hipGetLastError());
  tm.mark(1, s);
  HIP_TRY(spin_sync(s));
  g_view_ms = tm.ok ? tm.span(0, 1) : 0.0;
  t->bu_frames = std::move(f_out);
  t->bu_excl = std::move(e_out);
  t->bu_incl = std::move(i_out);
  t->bu_k = G;
  return CCT_OK;
}

}  // namespace

cct_status cct_bottom_up(cct_tree *tree, void *hip_stream, int64_t capacity, uint32_t *frames, uint64_t *excl,
                         uint64_t *incl, int64_t *n_frames) {
  clear_error();
  if (!tree || !n_frames) return fail(CCT_EINVAL, "NULL argument");
  if (capacity < 0) return fail(CCT_EINVAL, "negative capacity");
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  hipStream_t s = (hipStream_t)hip_stream;
  AllocHook hook;
  if (tree->bu_k < 0) {
    cct_status st = compute_bottom_up(tree, s);
    if (st) return st;
  }
  const int64_t K = tree->bu_k;
  if (K > 0 && capacity >= K) {
    const size_t m = (size_t)tree->m;
    if (frames) HIP_TRY(hipMemcpyAsync(frames, tree->bu_frames.p, (size_t)K * 4, hipMemcpyDefault, s));
    if (excl) HIP_TRY(hipMemcpyAsync(excl, tree->bu_excl.p, (size_t)K * m * 8, hipMemcpyDefault, s));
    if (incl) HIP_TRY(hipMemcpyAsync(incl, tree->bu_incl.p, (size_t)K * m * 8, hipMemcpyDefault, s));
    HIP_TRY(spin_sync(s));
  }
  *n_frames = K;
  return CCT_OK;
}

}  // extern "C"

namespace {

// Checks shared by both filter entry points; fills a.
cct_status filter_args(const cct_tree *tree, const cct_filter_spec *spec, int64_t capacity, const int64_t *node_ids,
                       const int64_t *n_matches, FilterArgs &a) {
  if (!tree || !spec || !n_matches) return fail(CCT_EINVAL, "NULL argument");
  if (capacity < 0 || (capacity > 0 && !node_ids)) return fail(CCT_EINVAL, "bad output capacity");
  const int32_t m = tree->m;
  if (spec->num_metric < 0 || spec->num_metric >= m) return fail(CCT_EINVAL, "num_metric out of range");
  if (spec->den_kind < kDenOne || spec->den_kind > kDenRoot) return fail(CCT_EINVAL, "unknown den_kind");
  if (spec->den_kind != kDenOne && (spec->den_metric < 0 || spec->den_metric >= m))
    return fail(CCT_EINVAL, "den_metric out of range");
  if (spec->op != 1 && spec->op != -1) return fail(CCT_EINVAL, "op must be +1 or -1");
  if (spec->thr_den == 0) return fail(CCT_EINVAL, "thr_den is 0");
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  a = FilterArgs{};
  a.u = tree->u; a.m = m; a.excl = tree->excl.as<uint64_t>(); a.incl = tree->incl.as<uint64_t>();
  a.subend = tree->subend.as<uint32_t>();
  a.num_metric = spec->num_metric; a.num_excl = spec->num_excl != 0;
  a.den_kind = spec->den_kind; a.den_metric = spec->den_metric; a.den_excl = spec->den_excl != 0;
  a.op = spec->op; a.thr_num = spec->thr_num; a.thr_den = spec->thr_den; a.leaves_only = spec->leaves_only != 0;
  return CCT_OK;
}

// The filter's three passes over the given scratch; the match count is copied to *dst
// (host memory) and the stream synchronised.
cct_status run_filter(const FilterArgs &a, const FilterScratch &f, int64_t capacity, int64_t *node_ids,
                      unsigned long long *dst, hipStream_t s) {
  const int64_t T = filter_tiles(a.u);
  launch_filter_mask(a, f.mask, f.count, s);
  launch_filter_scan(f.count, T, f.pos, s);
  launch_filter_write(a.u, f.mask, f.pos, capacity, node_ids, s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(dst, f.pos + T, 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));  // blocking: cct_filter_noalloc shares this path and creates no event
  return CCT_OK;
}

}  // namespace

extern "C" {

cct_status cct_filter(const cct_tree *tree, const cct_filter_spec *spec, void *hip_stream, int64_t capacity,
                      int64_t *node_ids, int64_t *n_matches) {
  AllocHook hook;
  clear_error();
  FilterArgs a;
  cct_status st = filter_args(tree, spec, capacity, node_ids, n_matches, a);
  if (st) return st;
  hipStream_t s = (hipStream_t)hip_stream;
  unsigned long long *hs = host_scratch();
  if (!hs) return fail(CCT_ENOMEM, "pinned host allocation failed");
  const int64_t T = filter_tiles(a.u);
  Buf mask, count, pos;
  if (!mask.alloc(T * (kFilterTile / 64) * 8) || !count.alloc(T * 4) || !pos.alloc((T + 1) * 8))
    return fail(CCT_ENOMEM, "device allocation failed");
  FilterScratch f{mask.as<uint64_t>(), count.as<uint32_t>(), pos.as<uint64_t>()};
  Timer tm;
  tm.mark(0, s);
  st = run_filter(a, f, capacity, node_ids, hs, s);
  if (st) return st;
  tm.mark(1, s);
  g_filter_ms = tm.ok ? tm.span(0, 1) : 0.0;
  *n_matches = (int64_t)hs[0];
  return CCT_OK;
}

cct_status cct_filter_noalloc(const cct_tree *tree, const cct_filter_spec *spec, void *hip_stream, int64_t capacity,
                              int64_t *node_ids, int64_t *n_matches) {
  clear_error();
  FilterArgs a;
  cct_status st = filter_args(tree, spec, capacity, node_ids, n_matches, a);
  if (st) return st;
  if (filter_tiles(a.u) > kFilterStaticTiles)
    return fail(CCT_EOVERFLOW, "tree has more nodes than cct_filter_noalloc's scratch holds (31,457,280)");
  void *base = filter_static_scratch();
  if (!base) return fail(CCT_EDEVICE, "address of the static filter scratch not available");
  unsigned long long k = 0;  // pageable: no pinned staging is allocated
  st = run_filter(a, filter_static_layout(base), capacity, node_ids, &k, (hipStream_t)hip_stream);
  if (st) return st;
  *n_matches = (int64_t)k;
  return CCT_OK;
}

cct_status cct_stats(const cct_tree *tree, void *hip_stream, const cct_node_stats *out) {
  AllocHook hook;
  clear_error();
  if (!tree || !out) return fail(CCT_EINVAL, "NULL argument");
  if (!tree->stats) return fail(CCT_EINVAL, "the tree keeps no statistics (build it with cct_build_stats)");
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  hipStream_t s = (hipStream_t)hip_stream;
  const int32_t m = tree->m;
  const int64_t U = tree->u, D = tree->d, C = 1 + 4 * (int64_t)m;
  const int64_t nblk = std::max<int64_t>(rmq_blocks(D), 1);
  const int levels = floor_log2((uint64_t)nblk) + 1;
  Buf rows, prefix, blk, node_path, cmin, pre, suf, tab;
  if (!rows.alloc(D * C * 8) || !prefix.alloc((D + 1) * C * 8) || !blk.alloc((D / 1024 + 2) * C * 8) ||
      !node_path.alloc(U * 4) || !cmin.alloc(D * m * 8) || !pre.alloc(D * m * 8) || !suf.alloc(D * m * 8) ||
      !tab.alloc(levels * nblk * m * 8))
    return fail(CCT_ENOMEM, "device allocation failed");
  NodeStatArgs a{};
  a.u = U; a.d = tree->d; a.m = m;
  a.scan_out = tree->scan_out.as<uint64_t>(); a.order = tree->order.as<uint32_t>();
  a.pcnt = tree->pcnt.as<uint64_t>(); a.pmin = tree->pmin.as<uint64_t>(); a.psq = tree->psq.as<uint64_t>();
  a.subend = tree->subend.as<uint32_t>(); a.excl = tree->excl.as<uint64_t>(); a.incl = tree->incl.as<uint64_t>();
  a.rows = rows.as<uint64_t>(); a.prefix = prefix.as<uint64_t>(); a.node_path = node_path.as<uint32_t>();
  a.cmin = cmin.as<uint64_t>();
  a.pre = pre.as<uint64_t>(); a.suf = suf.as<uint64_t>(); a.tab = tab.as<uint64_t>();
  a.nblk = nblk; a.levels = levels;
  a.out = NodeStatOut{out->count_excl, out->count_incl, out->min_excl, out->min_incl, out->sumsq_excl,
                      out->sumsq_incl, out->mean_excl, out->mean_incl, out->std_excl, out->std_incl};
  Timer tm;
  tm.mark(0, s);
  launch_node_stats(a, blk.as<uint64_t>(), s);
  tm.mark(1, s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(spin_sync(s));
  g_node_stats_ms = tm.ok ? tm.span(0, 1) : 0.0;
  return CCT_OK;
}

cct_status cct_query(const cct_tree *tree, const cct_paths *q, void *hip_stream, int64_t *node_ids, uint64_t *excl,
                     uint64_t *incl) {
  clear_error();
  if (!tree || !q) return fail(CCT_EINVAL, "NULL argument");
  if (q->n_events < 0 || q->n_frames < 0 || !q->offsets || (q->n_frames > 0 && !q->frames))
    return fail(CCT_EINVAL, "bad query batch");
  if (q->n_events > CCT_MAX_EVENTS) return fail(CCT_EOVERFLOW, "too many queries in one call");
  if (q->n_events > 0 && !node_ids) return fail(CCT_EINVAL, "node_ids is NULL");
  if (((uintptr_t)q->offsets & 7) || ((uintptr_t)q->frames & 3) || ((uintptr_t)node_ids & 7) ||
      ((uintptr_t)excl & 7) || ((uintptr_t)incl & 7))
    return fail(CCT_EINVAL, "misaligned pointer");
  if (q->n_events == 0) return CCT_OK;
  int dev = 0;
  (void)hipGetDevice(&dev);
  if (dev != tree->device) return fail(CCT_EINVAL, "tree belongs to another device");
  hipStream_t s = (hipStream_t)hip_stream;
  unsigned long long *hs = host_scratch();
  if (!hs) return fail(CCT_ENOMEM, "pinned host allocation failed");
  g_alloc_countdown = 0;  // queries allocate only what the index needs; the hook is not armed
  Buf err;
  if (!err.alloc(8)) return fail(CCT_ENOMEM, "device allocation failed");
  QueryArgs a{};
  a.q = q->n_events; a.qn_frames = q->n_frames; a.qoff = q->offsets; a.qfr = q->frames;
  a.d = tree->d; a.u = tree->u; a.m = tree->m;
  a.pframes = tree->pframes.as<uint32_t>(); a.pstart = tree->pstart.as<int64_t>(); a.plen = tree->plen.as<uint32_t>();
  a.order = tree->order.as<uint32_t>(); a.lcp = tree->lcp.as<uint32_t>(); a.scan_out = tree->scan_out.as<uint64_t>();
  a.excl = tree->excl.as<uint64_t>(); a.incl = tree->incl.as<uint64_t>();
  a.node_ids = node_ids; a.qexcl = excl; a.qincl = incl; a.err = err.as<unsigned long long>();
  // the batch's offsets are checked before anything is written to the outputs
  HIP_TRY(hipMemsetAsync(err.p, 0, 8, s));
  launch_query_check(a, s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(hs, err.p, 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(spin_sync(s));
  if (hs[0]) return fail(CCT_EINVAL, "malformed query offsets");
  // the index: every node under the hash of its prefix (a test setting keeps fewer key bits,
  // forcing collisions, on trees of at most 2^15 nodes: on larger ones a few keys would
  // make probing quadratic; another one uses the binary search); a table at most half full
  const int qbits = tree->u <= (1 << 15) ? (int)env_int("CCT_TEST_QUERY_HASH_BITS", 64) : 64;
  const uint64_t hash_mask = qbits >= 64 ? ~0ull : ((1ull << (qbits < 1 ? 1 : qbits)) - 1);
  const bool use_index = !env_int("CCT_TEST_QUERY_SEARCH", 0);
  g_qindex_ms = 0;
  if (!tree->q_ready || tree->q_hash_mask != hash_mask || (tree->q_cap != 0) != use_index) {
    tree->q_ready = false;
    Timer ti;
    ti.mark(0, s);
    if (!tree->q_sorted.alloc((size_t)std::max<int64_t>(tree->d, 1) * 16))
      return fail(CCT_ENOMEM, "device allocation failed");
    a.sorted = tree->q_sorted.as<int64_t>();
    launch_sorted_paths(a, s);
    tree->q_cap = 0;
    tree->q_tab.release();
    const uint64_t cap = pow2_at_least((uint64_t)std::max<int64_t>(2 * tree->u, 64));
    if (use_index && tree->q_tab.alloc(cap * 16)) {  // without room for it, the binary search
      tree->q_cap = cap;
      HIP_TRY(hipMemsetAsync(tree->q_tab.p, 0, cap * 16, s));
      a.qtab = tree->q_tab.as<uint64_t>(); a.qcap_mask = cap - 1; a.qhash_mask = hash_mask;
      launch_query_index(a, s);
    }
    ti.mark(1, s);
    HIP_TRY(hipGetLastError());
    HIP_TRY(spin_sync(s));
    g_qindex_ms = ti.ok ? ti.span(0, 1) : 0.0;
    tree->q_hash_mask = hash_mask;
    tree->q_ready = true;
  }
  a.sorted = tree->q_sorted.as<int64_t>();
  if (tree->q_cap) {
    a.qtab = tree->q_tab.as<uint64_t>(); a.qcap_mask = tree->q_cap - 1; a.qhash_mask = hash_mask;
  }
  Timer tm;
  tm.mark(0, s);
  launch_query(a, s);
  tm.mark(1, s);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync(hs, err.p, 8, hipMemcpyDeviceToHost, s));
  HIP_TRY(spin_sync(s));
  g_query_ms = tm.ok ? tm.span(0, 1) : 0.0;
  if (hs[0] & 2) return fail(CCT_EDEVICE, "query found an inconsistent tree");
  if (hs[0]) return fail(CCT_EINVAL, "malformed query offsets");
  return CCT_OK;
}

cct_status cct_info(const cct_tree *tree, int64_t *n_nodes, int32_t *n_metrics, int64_t *n_paths) {
  if (!tree) return fail(CCT_EINVAL, "tree is NULL");
  if (n_nodes) *n_nodes = tree->u;
  if (n_metrics) *n_metrics = tree->m;
  if (n_paths) *n_paths = tree->d;
  return CCT_OK;
}

cct_status cct_export(const cct_tree *tree, void *hip_stream, uint32_t *parent, uint32_t *frame, uint32_t *depth,
                      uint64_t *excl, uint64_t *incl) {
  clear_error();
  if (!tree) return fail(CCT_EINVAL, "tree is NULL");
  hipStream_t s = (hipStream_t)hip_stream;
  const size_t U = (size_t)tree->u, m = (size_t)tree->m;
  if (parent) HIP_TRY(hipMemcpyAsync(parent, tree->parent.p, U * 4, hipMemcpyDefault, s));
  if (frame) HIP_TRY(hipMemcpyAsync(frame, tree->frame.p, U * 4, hipMemcpyDefault, s));
  if (depth) HIP_TRY(hipMemcpyAsync(depth, tree->depth.p, U * 4, hipMemcpyDefault, s));
  if (excl) HIP_TRY(hipMemcpyAsync(excl, tree->excl.p, U * m * 8, hipMemcpyDefault, s));
  if (incl) HIP_TRY(hipMemcpyAsync(incl, tree->incl.p, U * m * 8, hipMemcpyDefault, s));
  HIP_TRY(spin_sync(s));
  return CCT_OK;
}

void cct_free(cct_tree *tree) { delete tree; }

void cct_release_cached_memory(void) {
  Pool &P = pool();
  std::lock_guard<std::mutex> lk(P.mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (auto &kv : P.cache) {
    (void)hipSetDevice(kv.first.first);
    (void)hipFree(kv.second);
  }
  P.cache.clear();
  (void)hipSetDevice(cur);
  (void)hipGetLastError();
}

const char *cct_last_error(void) { return g_error; }

int cct_last_timings(double *ms, int n) {
  if (!ms || n <= 0) return 0;
  const int k = n < 12 ? n : 12;
  for (int i = 0; i < k && i < 5; ++i) ms[i] = g_timings[i];
  if (k > 5) ms[5] = g_join_ms;
  if (k > 6) ms[6] = g_view_ms;
  if (k > 7) ms[7] = g_filter_ms;
  if (k > 8) ms[8] = g_stats_ms;
  if (k > 9) ms[9] = g_node_stats_ms;
  if (k > 10) ms[10] = g_query_ms;
  if (k > 11) ms[11] = g_qindex_ms;
  return k;
}

}  // extern "C"
