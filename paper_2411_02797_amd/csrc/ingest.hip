// Ingest: one HBM pass over a CSR batch of call paths that validates the offsets,
// hashes every path, maps it exactly onto its distinct full path in the unique-path
// table, and sums its metrics into that path's exclusive sums.
//
// This is the "insert call paths, collapse frames that refer to the same location"
// and "aggregate metrics within the same context" step of the profiler (Design,
// "Profiler", "Calling Context Tree"; Overview), done once per distinct full path
// instead of once per event and per frame: two events land on the same table entry
// iff their paths are equal frame by frame, which is exactly when the paper's tree
// insertion would end them on the same node.
//
// Work decomposition: one workgroup of 16 waves per CU, persistent.  Every wave owns a
// contiguous range of events and cuts it into tiles that fill its 1024-frame LDS
// slice (at most 63 events: lane j holds offset j), without workgroup barriers, so a
// CU keeps 16 tiles in flight.  While a wave resolves tile t, the frames of tile t+1
// stream into registers.  Lane l holds the 16-byte groups l, l + 64, l + 128,
// l + 192 of a tile, so every load instruction reads 1 KiB of consecutive frames
// (fully coalesced HBM stream) and every LDS access of a wave hits distinct banks.
//   - hash: each lane sums a position-dependent term over its four runs of four
//     frames; partial sums per event meet in LDS (64-bit LDS atomics).  The hash is a
//     sum of terms, so partial sums over any split of a path combine by adding.  The
//     walk also records each frame's event.
//   - dedup: lane j resolves event j: a path with the same hash and length already
//     resolved in this workgroup (LDS cache), else the table (linear probing, one
//     64-bit CAS claims an empty slot).  Every candidate is verified frame by frame:
//     lane l compares staged frames l, l + 64, ... with the candidate's frames, so
//     each load instruction reads 64 consecutive frames (L2/MALL resident: hot paths
//     are few).
//   - metrics: summed into the cache entry of the path (LDS atomics) and flushed to
//     HBM with 64-bit atomics once per workgroup; paths outside the cache add to HBM
//     directly.
#include "common.h"

namespace cct {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
enum : int32_t { kProbing = 0, kCandidate = 1, kResolved = 2, kFailed = 3 };
enum : int32_t { kTileFast = 0, kTileSlow = 1, kTileBad = 2, kTileNone = 3 };

constexpr int kWaves = kIngestThreads / 64;
constexpr uint32_t kNotReady = 0xFFFFFFFFu;
constexpr uint64_t kInStore = 1ull << 63;   // cache cbase: frames live in the path store

struct WaveShared {
  uint32_t fr[kWaveFrames];        // staged frames: slot x <-> relative position x - lead
  uint8_t evt[kWaveFrames];        // event of each staged slot
  int32_t ls[kWaveEvents + 1];     // event starts relative to the tile's first frame
  int32_t bad[kWaveEvents + 1];    // verification found a differing frame
  uint64_t hacc[kWaveEvents + 1];  // hash partial sums
  uint64_t vaddr[kWaveEvents + 1]; // byte address of the candidate frame at relative position 0, or 0
};

// Per-workgroup cache of resolved paths, keyed by (hash, length): the table slot,
// where that slot's frames live (to verify against) and this workgroup's metric sums
// for it.  Hot paths cost no table access after their first resolution in a
// workgroup, and one global atomic per metric per workgroup at the end.
struct IngestShared {
  uint64_t ckey[kCacheEntries];    // hash (0: empty / not cacheable)
  uint64_t cbase[kCacheEntries];   // first frame (kInStore: in the path store)
  uint32_t clen[kCacheEntries];
  uint32_t cslot[kCacheEntries];   // kNotReady until the entry is filled in
  uint64_t csum[kCacheWords];      // [entries][m]
  WaveShared wv[kWaves];
};

__device__ inline void wave_sync() {
  // orders this wave's LDS accesses: every lane's earlier LDS writes are visible to
  // every lane's later LDS reads
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_wave_barrier();
}

__device__ inline int cache_entries(int m) {
  int e = kCacheWords / m;
  if (e > kCacheEntries) e = kCacheEntries;
  int p = 1;
  while (p * 2 <= e) p *= 2;
  return p;
}

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, o, 64), hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

// wave-uniform values kept in scalar registers
__device__ inline int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ inline int64_t shfl_i64(int64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src, 64), hi = __shfl((uint32_t)((uint64_t)v >> 32), src, 64);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// A tile: events [e0, e0 + ne) of the wave's range, wave-uniform.
struct Tile {
  int64_t e0, g0;
  int32_t ne, span, lead, kind;
};

// Offsets window at event e (lane j holds offsets[e + j], j <= min(63, end - e)).
__device__ inline int64_t load_window(const IngestArgs &a, int64_t e, int64_t end, int lane) {
  return e < end && lane <= end - e ? a.off[e + lane] : 0;
}

// Validate the window and cut the next tile: as many events as fit in the staging
// slice.  Every offset is validated here, before any frame is read.
__device__ inline Tile make_tile(const IngestArgs &a, int64_t e, int64_t end, int64_t o, int lane) {
  Tile t{};
  if (e >= end) { t.kind = kTileNone; return t; }
  t.e0 = e;
  const int jmax = (int)min((int64_t)kWaveEvents, end - e);
  const int64_t onext = shfl_i64(o, lane + 1 < 64 ? lane + 1 : 63);
  bool bad = lane < jmax && onext < o;
  if (lane <= jmax) bad |= o < 0 || o > a.n_frames;
  if (lane == 0) bad |= e == 0 && o != 0;
  if (lane == jmax) bad |= e + jmax == a.n_events && o != a.n_frames;
  if (__any(bad)) { t.kind = kTileBad; return t; }
  t.g0 = uniform64(shfl_i64(o, 0));
  t.lead = (int)(((uintptr_t)a.fr >> 2) + (uint64_t)t.g0) & 3;
  const uint64_t fit = __ballot(lane >= 1 && lane <= jmax && o - t.g0 + t.lead <= kWaveFrames);
  if (fit == 0) {  // a single path longer than the slice
    t.ne = 1;
    t.kind = kTileSlow;
    return t;
  }
  t.ne = 63 - __builtin_clzll(fit);  // offsets are non-decreasing: the fitting lanes are 1..ne
  t.span = (int)(uniform64(shfl_i64(o, t.ne)) - t.g0);
  t.kind = kTileFast;
  return t;
}

// This lane's frames of a fast tile: 16-byte groups q * 64 + lane (slots
// 256 q + 4 lane .. + 4), at 16-byte aligned addresses; elements outside the tile are
// left zero.
__device__ inline void load_frames(const IngestArgs &a, const Tile &t, int lane, u32x4 nf[4]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = q * 256 + lane * 4 - t.lead;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (t.kind == kTileFast && r + 4 > 0 && r < t.span) {
      const int64_t gi = t.g0 + r;
      if (gi >= 0 && gi + 4 <= a.n_frames) {
        v = __builtin_nontemporal_load((const u32x4 *)(a.fr + gi));
      } else {
        for (int e = 0; e < 4; ++e)
          if (r + e >= 0 && r + e < t.span) v[e] = a.fr[gi + e];
      }
    }
    nf[q] = v;
  }
}

// Per-event resolution state, held by the lane that owns the event.
struct Probe {
  uint64_t h;        // final hash (masked)
  uint64_t cbase;    // frames of the candidate / resolved path (kInStore bit: path store)
  uint32_t slot;     // current probe slot (capacity <= 2^31)
  uint32_t steps;    // slots probed so far
  uint32_t len;      // staged events are shorter than a tile
  int32_t state;
};

// Walk the probe sequence until the event claims an empty slot (resolved, new path)
// or meets a slot whose tag and length match (candidate, needs verification).
// Every event probes at most `capacity` slots over all its rounds: past the load
// limit the table may be full, and the event then gives up (overflow).  Slot words
// are read through the caches: a stale empty word only leads to a CAS, which sees the
// true word.
__device__ __forceinline__ void probe(const IngestArgs &a, Probe &p, int64_t ev, int64_t ev_start, int64_t len) {
  const uint32_t tag = (uint32_t)(p.h >> 32);
  for (;;) {
    if ((uint64_t)p.steps++ > a.cap_mask) {
      atomicOr(&a.ctr[kCtrOverflow], 1ull);
      p.state = kFailed;
      return;
    }
    uint64_t w = a.slot[p.slot];
    if (w == kEmptySlot) {
      const uint64_t mine = ((uint64_t)tag << 32) | (kEventRef | (uint32_t)ev);
      const uint64_t prev = atomicCAS((unsigned long long *)&a.slot[p.slot], (unsigned long long)kEmptySlot,
                                      (unsigned long long)mine);
      if (prev == kEmptySlot) {
        const unsigned long long k = atomicAdd(&a.ctr[kCtrNew], 1ull);
        if (k < a.max_new) a.new_slots[k] = (uint32_t)p.slot;
        else atomicOr(&a.ctr[kCtrOverflow], 1ull);
        atomicAdd(&a.ctr[kCtrNewFrames], (unsigned long long)len);
        p.cbase = (uint64_t)ev_start;
        p.state = kResolved;
        return;
      }
      w = prev;
    }
    if ((uint32_t)(w >> 32) == tag) {
      const uint32_t ref = (uint32_t)w;
      int64_t clen;
      uint64_t cbase;
      if (ref & kEventRef) {
        const int64_t e = ref & kRefMask;
        const int64_t s = a.off[e];
        clen = a.off[e + 1] - s;
        cbase = (uint64_t)s;
      } else {
        clen = a.plen[ref];
        cbase = (uint64_t)a.pstart[ref] | kInStore;
      }
      if (clen == len) {
        p.cbase = cbase;
        p.state = len == 0 ? kResolved : kCandidate;
        return;
      }
    }
    p.slot = (uint32_t)((p.slot + 1) & a.cap_mask);
  }
}

// Cache entry holding a resolved path with this hash and length, or -1.
__device__ inline int cache_find(const IngestShared &S, uint64_t h, uint32_t len, int entries) {
  if (h == 0) return -1;
  uint32_t k = (uint32_t)h & (uint32_t)(entries - 1);
  for (int t = 0; t < 8; ++t) {
    const uint64_t key = S.ckey[k];
    if (key == 0) return -1;
    if (key == h && S.cslot[k] != kNotReady && S.clen[k] == len) return (int)k;
    k = (k + 1) & (uint32_t)(entries - 1);
  }
  return -1;
}

// Cache entry for a path just resolved to `slot`: the existing entry for it, a new
// one, or -1 (window full, or an entry for the same hash is not ready / names
// another slot: the caller then adds its metrics straight to HBM).
__device__ inline int cache_insert(IngestShared &S, uint64_t h, uint32_t len, uint32_t slot, uint64_t cbase,
                                   int entries) {
  if (h == 0) return -1;
  uint32_t k = (uint32_t)h & (uint32_t)(entries - 1);
  for (int t = 0; t < 8; ++t) {
    const uint64_t prev = atomicCAS((unsigned long long *)&S.ckey[k], 0ull, (unsigned long long)h);
    if (prev == 0) {
      S.cbase[k] = cbase;
      S.clen[k] = len;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      S.cslot[k] = slot;
      return (int)k;
    }
    if (prev == h) {
      const uint32_t cs = S.cslot[k];
      if (cs == kNotReady) return -1;
      if (cs == slot) return (int)k;
      if (S.clen[k] == len) return -1;  // same hash and length, another path
    }
    k = (k + 1) & (uint32_t)(entries - 1);
  }
  return -1;
}

// Add one event's metric into its cache entry or straight into HBM.
__device__ inline void add_metric(const IngestArgs &a, IngestShared &S, int ci, uint64_t slot, int c, uint64_t v) {
  if (ci >= 0) atomicAdd((unsigned long long *)&S.csum[ci * a.m + c], (unsigned long long)v);
  else atomicAdd((unsigned long long *)&a.delta[slot * a.m + c], (unsigned long long)v);
}

// Tiles whose frames exceed a wave's staging capacity: one event at a time, the
// wave striding over its frames in HBM.
__device__ __forceinline__ void slow_wave_tile(const IngestArgs &a, int64_t e0, int ne, int64_t o) {
  const int lane = threadIdx.x & 63;
  for (int j = 0; j < ne; ++j) {
    const int64_t gs = shfl_i64(o, j), len = shfl_i64(o, j + 1) - gs;
    uint64_t acc = 0;
    for (int64_t k = lane; k < len; k += 64) acc += frame_term(a.fr[gs + k], (uint32_t)k);
    acc = wave_sum_u64(acc);
    Probe p{};
    p.h = finish_hash(acc, (uint64_t)len) & a.hash_mask;
    p.slot = (uint32_t)(p.h & a.cap_mask);
    p.len = (uint32_t)len;  // compared with candidate lengths below as 64-bit
    p.state = kProbing;
    for (;;) {
      if (lane == 0) probe(a, p, e0 + j, gs, len);
      const int state = __shfl(p.state, 0, 64);
      if (state != kCandidate) { p.state = state; break; }
      const uint64_t cb = (uint64_t)shfl_i64((int64_t)p.cbase, 0);
      const uint32_t *src = (cb & kInStore) ? a.pframes + (cb & ~kInStore) : a.fr + cb;
      bool mism = false;
      for (int64_t k = lane; k < len; k += 64) mism |= a.fr[gs + k] != src[k];
      if (__any(mism)) {
        if (lane == 0) { p.slot = (uint32_t)((p.slot + 1) & a.cap_mask); p.state = kProbing; }
      } else {
        p.state = kResolved;
        break;
      }
    }
    if (p.state == kResolved) {
      const uint64_t slot = (uint64_t)shfl_i64((int64_t)p.slot, 0);
      if (lane < a.m) atomicAdd((unsigned long long *)&a.delta[slot * a.m + lane],
                                (unsigned long long)a.w[(e0 + j) * a.m + lane]);
    }
  }
}

// Event j containing relative position r (largest j with ls[j] <= r; ls[ne] > r).
__device__ inline int event_at(const WaveShared &W, int ne, int r) {
  int lo = 0, hi = ne;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (W.ls[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(kIngestThreads) void ingest_kernel(IngestArgs a) {
  __shared__ IngestShared S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  WaveShared &W = S.wv[wave];
  const int m = a.m;
  const int entries = cache_entries(m);
  for (int i = tid; i < kCacheEntries; i += kIngestThreads) { S.ckey[i] = 0; S.cslot[i] = kNotReady; }
  for (int i = tid; i < kCacheWords; i += kIngestThreads) S.csum[i] = 0;
  __syncthreads();

  // this wave's events
  const int64_t waves_total = (int64_t)gridDim.x * kWaves, w = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t end = (w + 1) * a.n_events / waves_total;
  int64_t e_cur = w * a.n_events / waves_total;
  int64_t o_cur = load_window(a, e_cur, end, lane);
  Tile t = make_tile(a, e_cur, end, o_cur, lane);
  u32x4 nf[4];
  load_frames(a, t, lane, nf);

  for (int iter = 0; t.kind != kTileNone; ++iter) {
    // early exit after a table overflow (the host retries); checked now and then, as
    // every check is an uncached read of one hot address
    if ((iter & 63) == 63 && __atomic_load_n(&a.ctr[kCtrOverflow], __ATOMIC_RELAXED)) break;
    if (t.kind == kTileBad) {
      if (lane == 0) atomicOr(&a.ctr[kCtrError], (unsigned long long)kErrOffsets);
      break;  // the call fails; this wave's range cannot be cut further
    }
    const int64_t e_nxt = t.e0 + t.ne;
    if (t.kind == kTileSlow) {
      slow_wave_tile(a, t.e0, t.ne, o_cur);
      e_cur = e_nxt;
      o_cur = load_window(a, e_cur, end, lane);
      t = make_tile(a, e_cur, end, o_cur, lane);
      load_frames(a, t, lane, nf);
      continue;
    }
    const int ne = t.ne, span = t.span, lead = t.lead;
    const int64_t e0 = t.e0;
    const int nm = ne * m;
    // stage the current frames; the next offsets window and this tile's metrics are
    // on their way while the tile is hashed
#pragma unroll
    for (int q = 0; q < 4; ++q) *(u32x4 *)&W.fr[q * 256 + lane * 4] = nf[q];
    if (lane <= ne) W.ls[lane] = (int32_t)(o_cur - t.g0);
    if (lane < ne) W.hacc[lane] = 0;
    const int64_t o_nxt = load_window(a, e_nxt, end, lane);
    const uint64_t mv0 = lane < nm ? a.w[e0 * m + lane] : 0;
    const uint64_t mv1 = lane + 64 < nm ? a.w[e0 * m + lane + 64] : 0;
    wave_sync();

    // A2: hash.  Four runs of four frames per lane: slots 256 q + 4 lane .. + 4.
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r0 = q * 256 + lane * 4 - lead;
      if (r0 + 4 > 0 && r0 < span) {
        const u32x4 v = *(const u32x4 *)&W.fr[q * 256 + lane * 4];
        int cur = event_at(W, ne, r0 < 0 ? 0 : r0), cs = W.ls[cur], nx = W.ls[cur + 1];
        uint64_t acc = 0;
        uint32_t ev4 = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = r0 + i;
          const bool valid = r >= 0 && r < span;
          if (valid && r >= nx) {
            atomicAdd((unsigned long long *)&W.hacc[cur], (unsigned long long)acc);
            acc = 0;
            do { ++cur; } while (W.ls[cur + 1] <= r);
            cs = W.ls[cur];
            nx = W.ls[cur + 1];
          }
          if (valid) acc += frame_term(v[i], (uint32_t)(r - cs));
          ev4 |= (uint32_t)cur << (8 * i);
        }
        atomicAdd((unsigned long long *)&W.hacc[cur], (unsigned long long)acc);
        *(uint32_t *)&W.evt[q * 256 + lane * 4] = ev4;
      }
    }
    // the next tile's frames stream in while this tile resolves
    const Tile tn = make_tile(a, e_nxt, end, o_nxt, lane);
    load_frames(a, tn, lane, nf);
    wave_sync();

    // A3: exact dedup.  Lane j resolves event j: a cached resolution of the same hash
    // and length, else the table; every candidate is verified by all lanes.
    Probe p{};
    p.state = kResolved;
    int ci = -1;  // cache entry of the candidate (-2: a cached candidate failed)
    if (lane < ne) {
      p.len = (uint32_t)(W.ls[lane + 1] - W.ls[lane]);
      p.h = finish_hash(W.hacc[lane], (uint64_t)p.len) & a.hash_mask;
      p.slot = (uint32_t)(p.h & a.cap_mask);
      p.state = kProbing;
      ci = cache_find(S, p.h, p.len, entries);
      if (ci >= 0) {
        p.slot = S.cslot[ci];
        p.cbase = S.cbase[ci];
        p.state = p.len == 0 ? kResolved : kCandidate;
      }
    }
    for (;;) {
      if (p.state == kProbing) probe(a, p, e0 + lane, o_cur, (int64_t)p.len);
      if (!__any(p.state == kCandidate)) break;
      if (lane < ne) {
        uint64_t va = 0;
        if (p.state == kCandidate) {
          const uint32_t *src = (p.cbase & kInStore) ? a.pframes + (p.cbase & ~kInStore) : a.fr + p.cbase;
          va = (uint64_t)(uintptr_t)src - 4ull * (uint64_t)W.ls[lane];
        }
        W.vaddr[lane] = va;
        W.bad[lane] = 0;
      }
      wave_sync();
      // lane l checks staged slots l, l + 64, ...: 64 consecutive frames per load
#pragma unroll
      for (int i = 0; i < kWaveFrames / 64; ++i) {
        const int x = i * 64 + lane, r = x - lead;
        if (r >= 0 && r < span) {
          const int e = W.evt[x];
          const uint64_t va = W.vaddr[e];
          if (va && *(const uint32_t *)(uintptr_t)(va + 4ull * (uint64_t)r) != W.fr[x]) W.bad[e] = 1;
        }
      }
      wave_sync();
      if (p.state == kCandidate) {
        if (W.bad[lane]) {
          p.slot = (uint32_t)((p.slot + 1) & a.cap_mask);
          p.state = kProbing;
          ci = -2;
        } else {
          p.state = kResolved;
        }
      }
      wave_sync();
    }

    // exclusive aggregation into the cache entry of the path (HBM atomics when none)
    int mi = -3;  // -3: nothing to add
    if (lane < ne && p.state == kResolved) {
      if (ci == -1) ci = cache_insert(S, p.h, p.len, p.slot, p.cbase, entries);
      mi = ci < 0 ? -1 : ci;
    }
    const uint32_t myslot = p.slot;
    for (int q0 = 0; q0 < nm; q0 += 64) {  // uniform trip count: every lane takes part in the shuffles
      const int q = q0 + lane;
      const int j = min(q / m, ne - 1), c = q - j * m;
      const int mj = __shfl(mi, j, 64);
      const uint64_t sj = __shfl(myslot, j, 64);
      if (q < nm && mj != -3) {
        const uint64_t v = q < 64 ? mv0 : q < 128 ? mv1 : a.w[e0 * m + q];
        add_metric(a, S, mj, sj, c, v);
      }
    }
    e_cur = e_nxt;
    o_cur = o_nxt;
    t = tn;
  }

  // flush the cached sums
  __syncthreads();
  for (int k = tid; k < entries; k += kIngestThreads) {
    const uint32_t slot = S.cslot[k];
    if (S.ckey[k] == 0 || slot == kNotReady) continue;
    for (int j = 0; j < m; ++j) {
      const uint64_t v = S.csum[k * m + j];
      if (v) atomicAdd((unsigned long long *)&a.delta[(uint64_t)slot * m + j], (unsigned long long)v);
    }
  }
}

// Publish the paths first seen in this call: give each a path id, copy its frames
// into the tree's path store (16-frame aligned, zero tail), write its checkpoint
// hashes and exclusive sums, and point its table slot at the path id.  One wave per
// path.
__global__ __launch_bounds__(256) void publish_kernel(PublishArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  if (i >= a.n_new) return;
  const uint32_t s = a.new_slots[i];
  const uint64_t w = a.slot[s];
  const int64_t e = (int64_t)((uint32_t)w & kRefMask);
  const int64_t src = a.off[e], len = a.off[e + 1] - src;
  const int64_t rl = round_store(len);
  const int64_t start = a.store_used + (int64_t)a.starts[i];
  const int64_t id = a.d_old + i;
  for (int64_t k = lane; k < rl; k += 64) a.pframes[start + k] = k < len ? a.fr[src + k] : 0u;
  // checkpoint hashes: lane b sums block b of 16 frames; a wave prefix scan then
  // gives the prefix sums at every block boundary
  uint64_t carry = 0;
  const int64_t nblk = len / kStoreAlign;
  for (int64_t b0 = 0; b0 < nblk; b0 += 64) {
    const int64_t b = b0 + lane;
    uint64_t v = 0;
    if (b < nblk)
      for (int k = 0; k < kStoreAlign; ++k) {
        const int64_t p = b * kStoreAlign + k;
        v += frame_term(a.fr[src + p], (uint32_t)p);
      }
    for (int o = 1; o < 64; o <<= 1) {  // inclusive scan across the wave
      uint32_t lo = __shfl_up((uint32_t)v, o, 64), hi = __shfl_up((uint32_t)(v >> 32), o, 64);
      if (lane >= o) v += ((uint64_t)hi << 32) | lo;
    }
    v += carry;
    if (b < nblk) a.pcp[start / kStoreAlign + b] = finish_hash(v, (uint64_t)(b + 1) * kStoreAlign);
    uint32_t lo = __shfl((uint32_t)v, 63, 64), hi = __shfl((uint32_t)(v >> 32), 63, 64);
    carry = ((uint64_t)hi << 32) | lo;
  }
  if (lane == 0) {
    a.pstart[id] = start;
    a.plen[id] = (uint32_t)len;
    a.pslot[id] = s;
    a.slot[s] = (w & 0xFFFFFFFF00000000ull) | (uint64_t)id;
  }
  if (lane < a.m) a.psums[id * a.m + lane] = a.delta[(uint64_t)s * a.m + lane];
}

// Padded store length of every new path (input of the scan that places them).
__global__ void new_lengths_kernel(const int64_t *off, const uint64_t *slot, const uint32_t *new_slots, int64_t n,
                                   uint64_t *out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t e = (int64_t)((uint32_t)slot[new_slots[i]] & kRefMask);
  out[i] = (uint64_t)round_store(off[e + 1] - off[e]);
}

__global__ void fold_old_kernel(int64_t d_old, int32_t m, const uint32_t *pslot, const uint64_t *delta,
                                uint64_t *psums) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= d_old * m) return;
  const int64_t d = t / m, j = t - d * m;
  psums[t] += delta[(uint64_t)pslot[d] * m + j];
}

// Roll back every slot claimed in the current call (after an error or overflow).
__global__ void unclaim_kernel(uint64_t *slot, uint64_t cap) {
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= cap) return;
  const uint64_t w = slot[t];
  if (w != kEmptySlot && ((uint32_t)w & kEventRef)) slot[t] = kEmptySlot;
}

// Re-insert the stored paths into a larger, empty table (distinct paths: no
// verification needed, each claims the first empty slot of its probe sequence).
__global__ void rehash_kernel(const uint32_t *pframes, const int64_t *pstart, const uint32_t *plen, int64_t d,
                              uint64_t *slot, uint64_t cap_mask, uint64_t hash_mask, uint32_t *pslot) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= d) return;
  const int64_t st = pstart[id];
  const uint32_t len = plen[id];
  uint64_t acc = 0;
  for (uint32_t k = 0; k < len; ++k) acc += frame_term(pframes[st + k], k);
  const uint64_t h = finish_hash(acc, len) & hash_mask;
  const uint64_t word = (h & 0xFFFFFFFF00000000ull) | (uint64_t)id;
  uint64_t s = h & cap_mask;
  while (atomicCAS((unsigned long long *)&slot[s], (unsigned long long)kEmptySlot, (unsigned long long)word) !=
         kEmptySlot)
    s = (s + 1) & cap_mask;
  pslot[id] = (uint32_t)s;
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_ingest(const IngestArgs &a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(ingest_kernel, dim3(grid), dim3(kIngestThreads), 0, s, a);
}
void launch_new_lengths(const int64_t *off, const uint64_t *slot, const uint32_t *new_slots, int64_t n,
                        uint64_t *out, hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(new_lengths_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, off, slot, new_slots, n, out);
}
void launch_publish(const PublishArgs &a, hipStream_t s) {
  if (a.n_new <= 0) return;
  hipLaunchKernelGGL(publish_kernel, dim3(blocks_for(a.n_new * 64, 256)), dim3(256), 0, s, a);
}
void launch_fold_old(int64_t d_old, int32_t m, const uint32_t *pslot, const uint64_t *delta, uint64_t *psums,
                     hipStream_t s) {
  if (d_old <= 0) return;
  hipLaunchKernelGGL(fold_old_kernel, dim3(blocks_for(d_old * m, 256)), dim3(256), 0, s, d_old, m, pslot, delta,
                     psums);
}
void launch_unclaim(uint64_t *slot, uint64_t cap, hipStream_t s) {
  hipLaunchKernelGGL(unclaim_kernel, dim3(blocks_for((int64_t)cap, 256)), dim3(256), 0, s, slot, cap);
}
void launch_rehash(const uint32_t *pframes, const int64_t *pstart, const uint32_t *plen, int64_t d,
                   uint64_t *slot, uint64_t cap_mask, uint64_t hash_mask, uint32_t *pslot, hipStream_t s) {
  if (d <= 0) return;
  hipLaunchKernelGGL(rehash_kernel, dim3(blocks_for(d, 256)), dim3(256), 0, s, pframes, pstart, plen, d, slot,
                     cap_mask, hash_mask, pslot);
}

}  // namespace cct
