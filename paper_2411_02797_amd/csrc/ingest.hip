// Ingest: one HBM pass over a CSR batch of call paths that validates the offsets,
// hashes every path and maps it exactly onto its distinct full path in the
// unique-path table (one table slot per distinct path), then a second, light pass
// sums every event's metrics into its slot.
//
// This is the "insert call paths, collapse frames that refer to the same location"
// and "aggregate metrics within the same context" step of the profiler (Design,
// "Profiler", "Calling Context Tree"; Overview), done once per distinct full path
// instead of once per event and per frame: two events land on the same slot iff
// their paths are equal frame by frame, which is exactly when the paper's tree
// insertion would end them on the same node.
//
// Work decomposition of the hashing pass: one workgroup of 16 waves per CU,
// persistent.  Every wave owns a contiguous range of events and cuts it into tiles
// that fill its 1024-frame LDS slice (at most 63 events: lane j holds offset j),
// without workgroup barriers, so a CU keeps 16 tiles in flight.  While a wave
// resolves tile t, the frames of tile t+1 stream into registers.  Lane l holds the
// 16-byte groups l, l + 64, l + 128, l + 192 of a tile, so every load instruction
// reads 1 KiB of consecutive frames (a fully coalesced HBM stream) and every LDS
// access of a wave hits distinct banks.
//   - hash: each lane sums a position-dependent term over its four runs of four
//     frames; partial sums per event meet in LDS (64-bit LDS atomics).  The hash is a
//     sum of terms, so partial sums over any split of a path combine by adding.  The
//     walk also records each frame's event.
//   - dedup: lane j resolves event j: a path with the same hash and length already
//     resolved in this workgroup (LDS cache), else the table (linear probing over
//     16-byte slots that carry the candidate's location, so one round trip; one
//     64-bit CAS claims an empty slot).  Every candidate is verified frame by frame:
//     lane l compares staged frames l, l + 64, ... with the candidate's frames, so
//     each load instruction reads 64 consecutive frames (L2/MALL resident: hot paths
//     are few).
#include "common.h"

namespace cct {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
enum : int32_t { kProbing = 0, kCandidate = 1, kResolved = 2, kFailed = 3 };
enum : int32_t { kTileFast = 0, kTileSlow = 1, kTileBad = 2, kTileNone = 3 };

constexpr int kWaves = kIngestThreads / 64;
constexpr uint32_t kNotReady = 0xFFFFFFFFu;
constexpr uint64_t kInStore = 1ull << 63;   // candidate base: frames live in the path store
constexpr uint64_t kRelVerify = 1ull << 62, kRelStore = 1ull << 61, kRelBias = kWaveFrames;
constexpr uint64_t kRelMask = kRelStore - 1;

struct WaveShared {
  uint32_t fr[kWaveFrames];        // staged frames: slot x <-> relative position x - lead
  uint8_t evt[kWaveFrames];        // event of each staged slot
  uint8_t gmap[kWaveFrames / 4];   // event containing the first position of each 4-slot group
  int32_t ls[kWaveEvents + 1];     // event starts relative to the tile's first frame
  int32_t bad[kWaveEvents + 1];    // verification found a differing frame
  uint64_t hacc[kWaveEvents + 1];  // hash partial sums
  uint64_t vrel[kWaveEvents + 1];  // candidate frame index at relative position 0 (+ kRelBias), with
                                   // kRelVerify / kRelStore flags; 0: nothing to verify
};

// Per-workgroup cache of resolved paths, keyed by (hash, length): the table slot and
// where that slot's frames live (to verify against).  Hot paths cost no table access
// after their first resolution in a workgroup.
struct IngestShared {
  uint64_t ckey[kCacheEntries];    // hash (0: empty / not cacheable)
  uint64_t cbase[kCacheEntries];   // first frame (kInStore: in the path store)
  uint32_t clen[kCacheEntries];
  uint32_t cslot[kCacheEntries];   // kNotReady until the entry is filled in
  WaveShared wv[kWaves];
};

// Orders this wave's LDS accesses: every lane's earlier LDS writes are visible to
// every lane's later LDS reads.  Waits for LDS operations only (lgkmcnt), so global
// loads in flight keep streaming.
__device__ inline void wave_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
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
// Every event probes at most `capacity` slots over all its rounds: a full table makes
// the event give up (overflow; the host retries with a larger table).  Slots are read
// through the caches: a stale empty word only leads to a CAS, which sees the true
// word.
__device__ __forceinline__ void probe(const IngestArgs &a, Probe &p, int64_t ev, int64_t ev_start, int64_t len) {
  const uint32_t tag = (uint32_t)(p.h >> 32);
  for (;;) {
    if ((uint64_t)p.steps++ > a.cap_mask) {
      atomicOr(&a.ctr[kCtrOverflow], 1ull);
      p.state = kFailed;
      return;
    }
    Slot *sl = a.slot + p.slot;
    uint64_t w = sl->word, info = sl->info;
    if (w == kEmptySlot) {
      const uint64_t mine = ((uint64_t)tag << 32) | (kEventRef | (uint32_t)ev);
      const uint64_t prev = atomicCAS((unsigned long long *)&sl->word, (unsigned long long)kEmptySlot,
                                      (unsigned long long)mine);
      if (prev == kEmptySlot) {
        sl->info = make_info((uint64_t)ev_start, false, (uint64_t)len);
        p.cbase = (uint64_t)ev_start;
        p.state = kResolved;
        return;
      }
      w = prev;
      info = kEmptyInfo;
    }
    if ((uint32_t)(w >> 32) == tag) {
      int64_t clen;
      uint64_t cbase;
      if (info != kEmptyInfo && (info & kInfoLongLen) != kInfoLongLen) {
        clen = (int64_t)(info & kInfoLongLen);
        cbase = (info >> 24) | (((info >> 23) & 1) ? kInStore : 0);
      } else {
        const uint32_t ref = (uint32_t)w;
        if (ref & kEventRef) {
          const int64_t e = ref & kRefMask;
          const int64_t s = a.off[e];
          clen = a.off[e + 1] - s;
          cbase = (uint64_t)s;
        } else {
          clen = a.plen[ref];
          cbase = (uint64_t)a.pstart[ref] | kInStore;
        }
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
__device__ inline int cache_find(const IngestShared &S, uint64_t h, uint32_t len) {
  if (h == 0) return -1;
  uint32_t k = (uint32_t)h & (uint32_t)(kCacheEntries - 1);
  for (int t = 0; t < 8; ++t) {
    const uint64_t key = S.ckey[k];
    if (key == 0) return -1;
    if (key == h && S.cslot[k] != kNotReady && S.clen[k] == len) return (int)k;
    k = (k + 1) & (uint32_t)(kCacheEntries - 1);
  }
  return -1;
}

// Remember a path just resolved to `slot` (unless its probe window is full, or an
// entry for the same hash and length names another path).
__device__ inline void cache_insert(IngestShared &S, uint64_t h, uint32_t len, uint32_t slot, uint64_t cbase) {
  if (h == 0) return;
  uint32_t k = (uint32_t)h & (uint32_t)(kCacheEntries - 1);
  for (int t = 0; t < 8; ++t) {
    const uint64_t prev = atomicCAS((unsigned long long *)&S.ckey[k], 0ull, (unsigned long long)h);
    if (prev == 0) {
      S.cbase[k] = cbase;
      S.clen[k] = len;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // payload before the ready slot id
      S.cslot[k] = slot;
      return;
    }
    if (prev == h) {
      const uint32_t cs = S.cslot[k];
      if (cs == kNotReady || cs == slot || S.clen[k] == len) return;
    }
    k = (k + 1) & (uint32_t)(kCacheEntries - 1);
  }
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
    const uint32_t slot = (uint32_t)__shfl((int)p.slot, 0, 64);
    if (lane == 0) a.slot_of[e0 + j] = p.state == kResolved ? slot : kNoSlot;
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
  for (int i = tid; i < kCacheEntries; i += kIngestThreads) { S.ckey[i] = 0; S.cslot[i] = kNotReady; }
  __syncthreads();

  // this wave's events.  Pipeline: the offsets window of tile t+1 is loaded during
  // tile t-1, so tile t+1's frames can be requested as soon as tile t starts.
  const int64_t waves_total = (int64_t)gridDim.x * kWaves, w = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t end = (w + 1) * a.n_events / waves_total;
  int64_t o_cur = load_window(a, w * a.n_events / waves_total, end, lane);
  Tile t = make_tile(a, w * a.n_events / waves_total, end, o_cur, lane);
  u32x4 nf[4];
  load_frames(a, t, lane, nf);
  int64_t o_nxt = t.kind == kTileFast || t.kind == kTileSlow ? load_window(a, t.e0 + t.ne, end, lane) : 0;

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
      o_cur = o_nxt;
      t = make_tile(a, e_nxt, end, o_cur, lane);
      load_frames(a, t, lane, nf);
      o_nxt = t.kind == kTileFast || t.kind == kTileSlow ? load_window(a, t.e0 + t.ne, end, lane) : 0;
      continue;
    }
    const int ne = t.ne, span = t.span, lead = t.lead;
    const int64_t e0 = t.e0;
#pragma unroll
    for (int q = 0; q < 4; ++q) *(u32x4 *)&W.fr[q * 256 + lane * 4] = nf[q];
    // event starts, and the group map: the event containing the first position of
    // every 4-slot group.  Event j is written to the first group that starts at or
    // after it, by the last event to map there (one writer per byte); a running max
    // then fills the groups in between.
    *(uint32_t *)&W.gmap[lane * 4] = 0;
    if (lane <= ne) W.ls[lane] = (int32_t)(o_cur - t.g0);
    {
      const int g = ((int)(o_cur - t.g0) + lead + 3) >> 2;
      const int gn = __shfl_down(g, 1, 64);
      wave_sync();
      if (lane < ne) {
        W.hacc[lane] = 0;
        if (g < kWaveFrames / 4 && (lane == ne - 1 || gn != g)) W.gmap[g] = (uint8_t)lane;
      }
    }
    wave_sync();
    {
      const uint32_t pk = *(const uint32_t *)&W.gmap[lane * 4];
      uint32_t b0 = pk & 0xFF, b1 = max(b0, (pk >> 8) & 0xFF), b2 = max(b1, (pk >> 16) & 0xFF),
               b3 = max(b2, pk >> 24);
      uint32_t run = b3;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t u = __shfl_up(run, o, 64);
        if (lane >= o) run = max(run, u);
      }
      uint32_t before = __shfl_up(run, 1, 64);
      if (lane == 0) before = 0;
      b0 = max(b0, before); b1 = max(b1, before); b2 = max(b2, before); b3 = max(b3, before);
      *(uint32_t *)&W.gmap[lane * 4] = b0 | b1 << 8 | b2 << 16 | b3 << 24;
    }
    wave_sync();

    // A2: hash.  Four runs of four frames per lane: slots 256 q + 4 lane .. + 4.
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r0 = q * 256 + lane * 4 - lead;
      if (r0 + 4 > 0 && r0 < span) {
        const u32x4 v = *(const u32x4 *)&W.fr[q * 256 + lane * 4];
        int cur = W.gmap[q * 64 + lane], cs = W.ls[cur], nx = W.ls[cur + 1];
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
    wave_sync();

    // the next tile's frames, and the offsets window after it, stream in while this
    // tile resolves
    const Tile tn = make_tile(a, e_nxt, end, o_nxt, lane);
    load_frames(a, tn, lane, nf);
    const int64_t o_nn = tn.kind == kTileFast || tn.kind == kTileSlow ? load_window(a, tn.e0 + tn.ne, end, lane) : 0;

    // A3: exact dedup.  Lane j resolves event j: a cached resolution of the same hash
    // and length, else the table; every candidate is verified by all lanes.
    Probe p{};
    p.state = kResolved;
    bool cached = false;  // the candidate came from the cache (no re-insert needed)
    if (lane < ne) {
      p.len = (uint32_t)(W.ls[lane + 1] - W.ls[lane]);
      p.h = finish_hash(W.hacc[lane], (uint64_t)p.len) & a.hash_mask;
      p.slot = (uint32_t)(p.h & a.cap_mask);
      p.state = kProbing;
      const int ci = cache_find(S, p.h, p.len);
      if (ci >= 0) {
        p.slot = S.cslot[ci];
        p.cbase = S.cbase[ci];
        p.state = p.len == 0 ? kResolved : kCandidate;
        cached = true;
      }
    }
    for (;;) {
      if (p.state == kProbing) probe(a, p, e0 + lane, o_cur, (int64_t)p.len);
      if (!__any(p.state == kCandidate)) break;
      if (lane < ne) {
        uint64_t v = 0;
        if (p.state == kCandidate)
          v = kRelVerify | ((p.cbase & kInStore) ? kRelStore : 0) |
              ((p.cbase & ~kInStore) + kRelBias - (uint64_t)W.ls[lane]);
        W.vrel[lane] = v;
        W.bad[lane] = 0;
      }
      wave_sync();
      // lane l checks staged slots l, l + 64, ...: every load instruction reads 64
      // consecutive frames.  Addresses are formed without branches and the loads are
      // issued in two batches of eight, so a tile costs two round trips.
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        uint32_t cand[4];
        uint32_t act = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = (h * 4 + i) * 64 + lane, r = x - lead;
          const bool in = r >= 0 && r < span;
          const uint64_t v = W.vrel[W.evt[x] & kWaveEvents];  // slots outside the span hold stale events
          const bool chk = in && (v & kRelVerify);
          const uint32_t *src = (v & kRelStore) ? a.pframes : a.fr;
          cand[i] = 0;
          if (chk) cand[i] = src[(v & kRelMask) - kRelBias + (uint64_t)r];
          act |= (uint32_t)chk << i;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = (h * 4 + i) * 64 + lane;
          if (((act >> i) & 1u) && cand[i] != W.fr[x]) W.bad[W.evt[x]] = 1;
        }
      }
      wave_sync();
      if (p.state == kCandidate) {
        if (W.bad[lane]) {
          p.slot = (uint32_t)((p.slot + 1) & a.cap_mask);
          p.state = kProbing;
          cached = true;  // resolved past a cached path with the same hash: not cacheable
        } else {
          p.state = kResolved;
        }
      }
      wave_sync();
    }
    if (lane < ne) {
      if (p.state == kResolved && !cached) cache_insert(S, p.h, p.len, p.slot, p.cbase);
      a.slot_of[e0 + lane] = p.state == kResolved ? p.slot : kNoSlot;
    }
    o_cur = o_nxt;
    o_nxt = o_nn;
    t = tn;
  }
}

// Metric sums per slot: one persistent workgroup per CU walks a contiguous event
// range and sums into an LDS map keyed by slot (a hot path costs one HBM atomic per
// metric per workgroup), falling back to HBM atomics when a key's probe window is
// full.  A key already in the map is found with plain LDS reads (broadcast), so hot
// keys cost no atomic compare-and-swap.
constexpr int kAggThreads = 1024;
constexpr int kAggWords = 16384;  // LDS sums (128 KiB)
constexpr int kAggKeys = 8192;
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;

__global__ __launch_bounds__(kAggThreads) void aggregate_kernel(const uint32_t *slot_of, const uint64_t *w, int64_t n,
                                                                int32_t m, uint64_t *delta) {
  __shared__ uint32_t key[kAggKeys];
  __shared__ uint64_t sum[kAggWords];
  const int tid = threadIdx.x;
  int entries = kAggWords / m;
  if (entries > kAggKeys) entries = kAggKeys;
  int p2 = 1;
  while (p2 * 2 <= entries) p2 *= 2;
  entries = p2;
  for (int i = tid; i < kAggKeys; i += kAggThreads) key[i] = kEmptyKey;
  for (int i = tid; i < kAggWords; i += kAggThreads) sum[i] = 0;
  __syncthreads();
  const int64_t b = blockIdx.x, nb = gridDim.x;
  const int64_t lo = b * n / nb, hi = (b + 1) * n / nb;
  for (int64_t e = lo + tid; e < hi; e += kAggThreads) {
    const uint32_t s = slot_of[e];
    if (s == kNoSlot) continue;
    uint32_t k = hash32(s) & (uint32_t)(entries - 1);
    int mi = -1;
    for (int t = 0; t < 8; ++t) {
      uint32_t cur = key[k];
      if (cur == kEmptyKey) cur = atomicCAS(&key[k], kEmptyKey, s);
      if (cur == kEmptyKey || cur == s) { mi = (int)k; break; }
      k = (k + 1) & (uint32_t)(entries - 1);
    }
    for (int j = 0; j < m; ++j) {
      const uint64_t v = w[e * m + j];
      if (mi >= 0) atomicAdd((unsigned long long *)&sum[mi * m + j], (unsigned long long)v);
      else atomicAdd((unsigned long long *)&delta[(uint64_t)s * m + j], (unsigned long long)v);
    }
  }
  __syncthreads();
  for (int k = tid; k < entries; k += kAggThreads) {
    const uint32_t s = key[k];
    if (s == kEmptyKey) continue;
    for (int j = 0; j < m; ++j) {
      const uint64_t v = sum[k * m + j];
      if (v) atomicAdd((unsigned long long *)&delta[(uint64_t)s * m + j], (unsigned long long)v);
    }
  }
}

// Slots claimed in this call: a block of 1024 threads scans 4096 slots, counts its
// claims, reserves list positions with one atomic, and writes them (the list order
// is irrelevant: paths get their canonical ids later).  Lengths come from the slot's
// info word; per-block sums of padded and exact lengths go to part[block][2].
constexpr int kCollectThreads = 1024, kCollectPerThread = 4;
__global__ __launch_bounds__(kCollectThreads) void collect_new_kernel(const Slot *slot, uint64_t cap,
                                                                      const int64_t *off, uint32_t *new_slots,
                                                                      unsigned long long *ctr,
                                                                      unsigned long long *part) {
  __shared__ uint32_t cnt;
  __shared__ unsigned long long base, frames, lens;
  if (threadIdx.x == 0) { cnt = 0; frames = 0; lens = 0; }
  __syncthreads();
  uint32_t found[kCollectPerThread], pos[kCollectPerThread];
  uint64_t my_frames = 0, my_lens = 0;
  int nf = 0;
  for (int r = 0; r < kCollectPerThread; ++r) {
    const uint64_t s = ((uint64_t)blockIdx.x * kCollectPerThread + r) * kCollectThreads + threadIdx.x;
    if (s >= cap) break;
    const Slot sl = slot[s];
    if (sl.word != kEmptySlot && ((uint32_t)sl.word & kEventRef)) {
      int64_t len;
      if (sl.info != kEmptyInfo && (sl.info & kInfoLongLen) != kInfoLongLen) {
        len = (int64_t)(sl.info & kInfoLongLen);
      } else {
        const int64_t e = (int64_t)((uint32_t)sl.word & kRefMask);
        len = off[e + 1] - off[e];
      }
      found[nf] = (uint32_t)s;
      pos[nf] = atomicAdd(&cnt, 1u);
      ++nf;
      my_frames += (uint64_t)round_store(len);
      my_lens += (uint64_t)len;
    }
  }
  if (nf) {
    atomicAdd(&frames, (unsigned long long)my_frames);
    atomicAdd(&lens, (unsigned long long)my_lens);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    base = cnt ? atomicAdd(&ctr[kCtrNew], (unsigned long long)cnt) : 0;
    part[blockIdx.x * 2] = frames;
    part[blockIdx.x * 2 + 1] = lens;
  }
  __syncthreads();
  for (int i = 0; i < nf; ++i) new_slots[base + pos[i]] = found[i];
}

// Totals of the per-block length sums into ctr (one block).
__global__ __launch_bounds__(256) void collect_sum_kernel(const unsigned long long *part, int64_t nblk,
                                                          unsigned long long *ctr) {
  __shared__ unsigned long long sf[256], sl[256];
  unsigned long long f = 0, l = 0;
  for (int64_t i = threadIdx.x; i < nblk; i += 256) { f += part[i * 2]; l += part[i * 2 + 1]; }
  sf[threadIdx.x] = f;
  sl[threadIdx.x] = l;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) { sf[threadIdx.x] += sf[threadIdx.x + o]; sl[threadIdx.x] += sl[threadIdx.x + o]; }
    __syncthreads();
  }
  if (threadIdx.x == 0) { ctr[kCtrNewFrames] = sf[0]; ctr[kCtrNewLen] = sl[0]; }
}

// Publish the paths first seen in this call: give each a path id, copy its frames
// into the tree's path store (16-frame aligned, zero tail), write its checkpoint
// hashes and exclusive sums, and point its table slot at the path id and the stored
// frames.  One wave per path.
__global__ __launch_bounds__(256) void publish_kernel(PublishArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  if (i >= a.n_new) return;
  const uint32_t s = a.new_slots[i];
  const uint64_t w = a.slot[s].word;
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
    a.slot[s].word = (w & 0xFFFFFFFF00000000ull) | (uint64_t)id;
    a.slot[s].info = make_info((uint64_t)start, true, (uint64_t)len);
  }
  if (lane < a.m) a.psums[id * a.m + lane] = a.delta[(uint64_t)s * a.m + lane];
}

// Padded store length of every new path (input of the scan that places them).
__global__ void new_lengths_kernel(const int64_t *off, const Slot *slot, const uint32_t *new_slots, int64_t n,
                                   uint64_t *out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t e = (int64_t)((uint32_t)slot[new_slots[i]].word & kRefMask);
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
__global__ void unclaim_kernel(Slot *slot, uint64_t cap) {
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= cap) return;
  const uint64_t w = slot[t].word;
  if (w != kEmptySlot && ((uint32_t)w & kEventRef)) {
    slot[t].word = kEmptySlot;
    slot[t].info = kEmptyInfo;
  }
}

// Re-insert the stored paths into a larger, empty table (distinct paths: no
// verification needed, each claims the first empty slot of its probe sequence).
__global__ void rehash_kernel(const uint32_t *pframes, const int64_t *pstart, const uint32_t *plen, int64_t d,
                              Slot *slot, uint64_t cap_mask, uint64_t hash_mask, uint32_t *pslot) {
  const int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= d) return;
  const int64_t st = pstart[id];
  const uint32_t len = plen[id];
  uint64_t acc = 0;
  for (uint32_t k = 0; k < len; ++k) acc += frame_term(pframes[st + k], k);
  const uint64_t h = finish_hash(acc, len) & hash_mask;
  const uint64_t word = (h & 0xFFFFFFFF00000000ull) | (uint64_t)id;
  uint64_t s = h & cap_mask;
  while (atomicCAS((unsigned long long *)&slot[s].word, (unsigned long long)kEmptySlot, (unsigned long long)word) !=
         kEmptySlot)
    s = (s + 1) & cap_mask;
  slot[s].info = make_info((uint64_t)st, true, len);
  pslot[id] = (uint32_t)s;
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_ingest(const IngestArgs &a, int grid, hipStream_t s) {
  hipLaunchKernelGGL(ingest_kernel, dim3(grid), dim3(kIngestThreads), 0, s, a);
}
void launch_aggregate(const uint32_t *slot_of, const uint64_t *w, int64_t n, int32_t m, uint64_t *delta, int grid,
                      hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(aggregate_kernel, dim3(grid), dim3(kAggThreads), 0, s, slot_of, w, n, m, delta);
}
int64_t collect_blocks(uint64_t cap) { return (int64_t)((cap + kCollectThreads * kCollectPerThread - 1) /
                                                         (kCollectThreads * kCollectPerThread)); }
void launch_collect_new(const Slot *slot, uint64_t cap, const int64_t *off, uint32_t *new_slots,
                        unsigned long long *ctr, unsigned long long *part, hipStream_t s) {
  const int64_t nb = collect_blocks(cap);
  hipLaunchKernelGGL(collect_new_kernel, dim3((unsigned)nb), dim3(kCollectThreads), 0, s, slot, cap, off, new_slots,
                     ctr, part);
  hipLaunchKernelGGL(collect_sum_kernel, dim3(1), dim3(256), 0, s, part, nb, ctr);
}
void launch_new_lengths(const int64_t *off, const Slot *slot, const uint32_t *new_slots, int64_t n, uint64_t *out,
                        hipStream_t s) {
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
void launch_unclaim(Slot *slot, uint64_t cap, hipStream_t s) {
  hipLaunchKernelGGL(unclaim_kernel, dim3(blocks_for((int64_t)cap, 256)), dim3(256), 0, s, slot, cap);
}
void launch_rehash(const uint32_t *pframes, const int64_t *pstart, const uint32_t *plen, int64_t d, Slot *slot,
                   uint64_t cap_mask, uint64_t hash_mask, uint32_t *pslot, hipStream_t s) {
  if (d <= 0) return;
  hipLaunchKernelGGL(rehash_kernel, dim3(blocks_for(d, 256)), dim3(256), 0, s, pframes, pstart, plen, d, slot,
                     cap_mask, hash_mask, pslot);
}

}  // namespace cct
