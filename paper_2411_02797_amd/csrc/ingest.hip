// Ingest: one HBM pass over a CSR batch of call paths that validates the offsets,
// hashes every path and maps it exactly onto its distinct full path in the
// unique-path table (one table slot per distinct path), then a second, light pass
// sums every event's metrics into its slot.
//
// This is the profiler's step that puts call paths into the tree, merging frames that
// name one location, and sums the metrics of equal contexts (Design, "Profiler",
// "Calling Context Tree"; Overview), done once per distinct full path
// instead of once per event and per frame: two events land on the same slot iff
// their paths are equal frame by frame, which is exactly when the paper's tree
// insertion would end them on the same node.
//
// Work decomposition of the hashing pass: one workgroup of 16 waves per CU,
// persistent.  Every wave owns a contiguous range of events and cuts it into tiles
// of at most 63 events whose paths, cut into blocks of 16 frames, fill at most 128
// blocks: lane l holds blocks l and l + 64 (16 consecutive frames of one event each)
// in registers, loaded with four 16-byte buffer loads per block (the buffer's range
// check makes reads past the end of the batch return zero).  Consecutive lanes hold
// consecutive blocks, so a wave's loads cover a contiguous stretch of the batch.
// Waves need no barriers, so a CU keeps 16 tiles in flight; a wave requests tile
// t+1's frames once tile t's table and candidate loads have returned.
//   - hash: a path's hash is a sum over its 16-frame blocks of terms of (pair of
//     frames, position in the path) (the last block of a path ends at the path's end);
//     a lane sums its block, and the block sums of an event meet in LDS.  A block
//     knows its position in the path, so no lane ever looks for an event boundary.
//   - dedup: lane j resolves event j: a path with the same hash and length already
//     resolved in this workgroup (LDS cache), else the table (linear probing over
//     16-byte slots that carry the candidate's location, so one round trip; one
//     64-bit CAS claims an empty slot).  Only the first lane of a workgroup to meet a
//     path probes the table for it; lanes that meet it meanwhile wait on its cache
//     entry, so a hot path is not claimed by thousands of CASes on one slot when every
//     wave meets it in its first tile.  Every candidate is verified frame by frame:
//     each block lane compares its 16 frames with the candidate's (16-byte loads; hot
//     candidates are L2 resident).
#include "common.h"

namespace cct {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef u32x4 u32x4_a4 __attribute__((aligned(4)));
// global-memory pointers (address space 1), so candidate loads are global loads
typedef const uint32_t __attribute__((address_space(1))) *gptr;
typedef const u32x4_a4 __attribute__((address_space(1))) *gptr4;
enum : int32_t { kProbing = 0, kCandidate = 1, kResolved = 2, kFailed = 3, kWaiting = 4 };
enum : int32_t { kTileFast = 0, kTileSlow = 1, kTileBad = 2, kTileNone = 3 };

constexpr int kWaves = kIngestThreads / 64;
constexpr int kBlock = 16;                        // frames per lane block
constexpr int kTileBlocks = kWaveFrames / kBlock;   // blocks per wave tile: kLaneBlocks per lane
constexpr uint32_t kNotReady = 0xFFFFFFFFu;  // cache entry claimed, its path not yet resolved
constexpr uint32_t kNoEntry = 0xFFFFFFFEu;   // cache entry's path could not be resolved (table full)
constexpr int kLeader = 1 << 16;              // added to a cache entry index: this lane claimed the entry
constexpr int kFromCache = -2;                // no entry; the lane's candidate came from the cache
constexpr uint64_t kInStore = 1ull << 63;   // candidate base: frames live in the path store

struct WaveShared {
  uint64_t hacc[64];  // hash sums per event
  uint64_t vptr[64];  // global address of the candidate's first frame; 0: nothing to verify
  uint32_t vlim[64];  // frames readable from vptr (the path, padded in the path store)
  uint8_t bad[64];    // verification found a differing frame
  uint8_t first[kTileBlocks];  // event whose first block is block b (0 if none)
};

// Per-workgroup cache of resolved paths, keyed by (hash, length): the table slot and
// where that slot's frames live (to verify against).  Hot paths cost no table access
// after their first resolution in a workgroup.  The first lane of the workgroup to miss on
// a key claims an entry for it and resolves the path in the table; lanes that meet the
// claimed entry meanwhile wait for it instead of probing the table themselves, so a path
// costs one table probe per workgroup however many of its events arrive together.
struct IngestShared {
  alignas(16) uint64_t ckey[kCacheEntries];  // hash (0: empty / not cacheable)
  uint64_t cbase[kCacheEntries];   // first frame (kInStore: in the path store)
  uint64_t cinfo[kCacheEntries];   // slot (low word; kNotReady until filled in), length (high)
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

// Inclusive scans over the 64 lanes (DPP row shifts, then row broadcasts).
template <bool kMax>
__device__ inline int wave_scan(int v) {
  auto op = [](int x, int y) { return kMax ? max(x, y) : x + y; };
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true));  // row_shr:1
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true));  // row_shr:2
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true));  // row_shr:4
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true));  // row_shr:8
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false)); // row_bcast:15
  v = op(v, __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false)); // row_bcast:31
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
  int64_t e0, g0;  // first event and its first frame
  int32_t ne, kind;
  int32_t span;    // frames of the tile's events
};

// One of this lane's blocks of a tile: frames [st, st + rem) of event ev (ev = -1: no
// block), the block of the path hash that starts at frame st (rem = 16 unless the path
// is shorter), at byte offset voff from the tile's first frame.  Lane l holds blocks
// l + 64 q, q < kLaneBlocks.
struct Blk {
  int32_t ev, st, rem, voff;
};

// This lane's index in the wave, computed afresh (two instructions) where a value kept
// in a register across the tile loop would be spilled.
__device__ inline int fresh_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Offsets window at event e (lane j holds offsets[e + j], j <= min(63, end - e); 0 past
// that).  A buffer load whose range ends at the window's last offset: the address lives in
// scalar registers, and lanes past the range read zero.
__device__ inline int64_t load_window(const IngestArgs &a, int64_t e, int64_t end, int lane) {
  if (e >= end) return 0;
  const int64_t eu = uniform64(e);
  const int bytes = __builtin_amdgcn_readfirstlane((int)(min(uniform64(end) - eu, (int64_t)63) + 1) * 8);
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void *)(a.off + eu), (short)0, bytes, 0x00020000);
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, fresh_lane() * 8, 0, 0);
  return (int64_t)(((uint64_t)v[1] << 32) | v[0]);
}

// Validate the window and cut the next tile: as many events as fit in the tile's
// blocks; map every lane to its blocks.  Every offset is validated here, before any
// frame is read.
__device__ inline Tile make_tile(const IngestArgs &a, WaveShared &W, int64_t e, int64_t end, int64_t o,
                                 Blk (&b)[kLaneBlocks]) {
  const int lane = fresh_lane();
  Tile t{};
#pragma unroll
  for (int q = 0; q < kLaneBlocks; ++q) b[q] = Blk{-1, 0, 0, 0};
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
  // blocks per event (kTileBlocks + 1: does not fit), inclusive prefix over events
  const int64_t len = lane < jmax ? onext - o : 0;
  const int nb = len > kWaveFrames ? kTileBlocks + 1 : (int)((len + kBlock - 1) / kBlock);
  const int incl = wave_scan<false>(nb);
  const uint64_t fit = __ballot(lane < jmax && incl <= kTileBlocks);
  t.ne = __popcll(fit);  // block counts are non-negative: the fitting events are a prefix
  if (t.ne == 0) {       // a single path longer than a tile
    t.ne = 1;
    t.kind = kTileSlow;
    return t;
  }
  t.kind = kTileFast;
  t.span = (int)(uniform64(shfl_i64(o, t.ne)) - t.g0);
  // block -> event: event j's blocks are [incl - nb, incl)
  const int nblk = __builtin_amdgcn_readlane(incl, t.ne - 1);
  const int excl = incl - nb;
  const int rel = (int)(o - t.g0);
#pragma unroll
  for (int q = 0; q < kLaneBlocks; ++q) W.first[q * 64 + lane] = 0;
  wave_sync();
  if (lane < t.ne && nb > 0) W.first[excl] = (uint8_t)lane;
  wave_sync();
  int carry = 0;
#pragma unroll
  for (int q = 0; q < kLaneBlocks; ++q) {
    const int ev = max(wave_scan<true>(W.first[q * 64 + lane]), carry);
    carry = __builtin_amdgcn_readlane(ev, 63);
    const int ev_excl = __shfl(excl, ev, 64);
    const int ev_len = __shfl((int)len, ev, 64);
    const int ev_start = __shfl(rel, ev, 64);
    const int bi = q * 64 + lane, m = bi - ev_excl;
    if (bi < nblk && m >= 0 && m * kBlock < ev_len) {
      const int st = (int)hash_block_start(m, ev_len);
      b[q] = Blk{ev, st, min(kBlock, ev_len - st), (ev_start + st) * 4};
    }
  }
  return t;
}

// Buffer resource over the batch's frames from the tile's first frame on: loads past
// the end of the batch return zero.
// The descriptor is wave-uniform; its words are read from the first lane so that the
// compiler keeps it in scalar registers (a descriptor it believes divergent costs a
// loop around every load).
__device__ inline __amdgpu_buffer_rsrc_t tile_rsrc(const IngestArgs &a, const Tile &t) {
  const int64_t g0 = uniform64(t.g0);
  const int64_t avail = a.n_frames - g0;
  const int bytes = __builtin_amdgcn_readfirstlane((int)(avail < (1 << 28) ? avail * 4 : (1 << 30)));
  return __builtin_amdgcn_make_buffer_rsrc((void *)(a.fr + g0), (short)0, bytes, 0x00020000);
}

// This lane's blocks: four 16-byte loads each; a 16-byte load that would reach past
// the end of the batch is split into 4-byte loads (each range checked).  Frames past a
// block's event are left as loaded (never used).
__device__ inline void load_blocks(const IngestArgs &a, const Tile &t, const Blk (&b)[kLaneBlocks],
                                   u32x4 (&nf)[kLaneBlocks][4]) {
  if (t.kind != kTileFast) return;
  const __amdgpu_buffer_rsrc_t r = tile_rsrc(a, t);
  const int64_t lim = (a.n_frames - t.g0) * 4;
  if ((int64_t)t.span * 4 + 64 <= lim) {
    // every load of the tile ends inside the batch: no per-lane conditions (idle
    // lanes and frames past a block's event read frames that are never used)
#pragma unroll
    for (int q = 0; q < kLaneBlocks; ++q)
#pragma unroll
      for (int j = 0; j < 4; ++j) nf[q][j] = __builtin_amdgcn_raw_buffer_load_b128(r, b[q].voff + 16 * j, 0, 0);
    return;
  }
#pragma unroll
  for (int q = 0; q < kLaneBlocks; ++q) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (4 * j < b[q].rem) {
        if (b[q].voff + 16 * j + 16 <= lim) {
          v = __builtin_amdgcn_raw_buffer_load_b128(r, b[q].voff + 16 * j, 0, 0);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            v[k] = __builtin_amdgcn_raw_buffer_load_b32(r, b[q].voff + 16 * j + 4 * k, 0, 0);
        }
      }
      nf[q][j] = v;
    }
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

// Look (hash, length) up in the cache.  The entries form aligned buckets of 8; a key
// lives in the bucket its hash names.  The bucket's 8 keys are read at once (four
// 16-byte LDS reads), so a lookup costs one LDS round trip plus one per entry it has to
// read or claim, instead of a chain of dependent reads along a probe sequence.
// Returns the entry index plus kLeader when this lane claimed a fresh entry (it resolves
// the path and fills the entry in), the entry index alone when an entry for the key
// exists (ready, or claimed and pending: the caller waits), or -1 when the key is not
// cacheable (hash 0, or its bucket holds no free entry and no entry for the key).
__device__ inline int cache_lookup(IngestShared &S, uint64_t h, uint32_t len) {
  if (h == 0) return -1;
  typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
  const int b0 = (int)((uint32_t)h & (uint32_t)(kCacheEntries / 8 - 1)) * 8;
  const u64x2 *kp = (const u64x2 *)&S.ckey[b0];
  uint32_t empty = 0, match = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const u64x2 v = kp[j];
    empty |= (v[0] == 0 ? 1u : 0u) << (2 * j) | (v[1] == 0 ? 1u : 0u) << (2 * j + 1);
    match |= (v[0] == h ? 1u : 0u) << (2 * j) | (v[1] == h ? 1u : 0u) << (2 * j + 1);
  }
  // entries are only ever filled in: a key seen is final, an empty one may have been taken
  for (uint32_t c = empty | match; c != 0; c &= c - 1) {
    const int t = __builtin_ctz(c), k = b0 + t;
    if ((empty >> t) & 1) {
      const uint64_t key = atomicCAS((unsigned long long *)&S.ckey[k], 0ull, (unsigned long long)h);
      if (key == 0) return k | kLeader;
      if (key != h) continue;
    }
    const uint64_t ci = S.cinfo[k];
    const uint32_t cs = (uint32_t)ci;
    if (cs == kNotReady || (cs != kNoEntry && (uint32_t)(ci >> 32) == len)) return k;
  }
  return -1;
}

// Fill in a claimed entry: payload first, then the slot that marks it ready.
__device__ inline void cache_fill(IngestShared &S, int k, uint32_t len, uint32_t slot, uint64_t cbase) {
  S.cbase[k] = cbase;
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  S.cinfo[k] = ((uint64_t)len << 32) | slot;
}

// Tiles whose frames exceed a wave's staging capacity: one event at a time, the
// wave striding over its frames in HBM.
__device__ __forceinline__ void slow_wave_tile(const IngestArgs &a, int64_t e0, int ne, int64_t o) {
  const int lane = fresh_lane();
  for (int j = 0; j < ne; ++j) {
    const int64_t gs = shfl_i64(o, j), len = shfl_i64(o, j + 1) - gs;
    uint64_t acc = 0;
    for (int64_t p = lane; p < 8 * ((len + kBlock - 1) / kBlock); p += 64) {  // (len > kWaveFrames: every block full)
      const int64_t f = gs + hash_block_start(p >> 3, len) + 2 * (p & 7);
      acc += pair_term(a.fr[f], a.fr[f + 1], (uint32_t)p);
    }
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


// Read by the verification of blocks that have no candidate, never written.
__device__ __attribute__((aligned(16))) uint32_t g_zero_block[kBlock];

__global__ __launch_bounds__(kIngestThreads) void ingest_kernel(IngestArgs a) {
  __shared__ IngestShared S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  WaveShared &W = S.wv[wave];
  for (int i = tid; i < kCacheEntries; i += kIngestThreads) { S.ckey[i] = 0; S.cinfo[i] = kNotReady; }
  __syncthreads();

  // this wave's events.  Pipeline: the offsets window of tile t+1 is loaded during
  // tile t-1, so tile t+1 can be cut as soon as tile t has resolved.
  const int64_t waves_total = (int64_t)gridDim.x * kWaves, w = (int64_t)blockIdx.x * kWaves + wave;
  const int64_t end = (w + 1) * a.n_events / waves_total;
  int64_t o_cur = load_window(a, w * a.n_events / waves_total, end, lane);
  Blk b[kLaneBlocks];
  Tile t = make_tile(a, W, w * a.n_events / waves_total, end, o_cur, b);
  u32x4 nf[kLaneBlocks][4];
  load_blocks(a, t, b, nf);
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
    // The four waves that share a SIMD take turns at the highest issue priority, one
    // tile each: with equal priorities the oldest wave always wins, the youngest falls
    // behind, and the SIMD ends with one wave and nothing to hide its latency behind.
    {
      const int r = (iter + __builtin_amdgcn_readfirstlane(wave >> 2)) & 3;
      if (r == 0) __builtin_amdgcn_s_setprio(0);
      else if (r == 1) __builtin_amdgcn_s_setprio(1);
      else if (r == 2) __builtin_amdgcn_s_setprio(2);
      else __builtin_amdgcn_s_setprio(3);
    }
    if (t.kind == kTileSlow) {
      slow_wave_tile(a, t.e0, t.ne, o_cur);
      o_cur = o_nxt;
      t = make_tile(a, W, e_nxt, end, o_cur, b);
      load_blocks(a, t, b, nf);
      o_nxt = t.kind == kTileFast || t.kind == kTileSlow ? load_window(a, t.e0 + t.ne, end, lane) : 0;
      continue;
    }
    const int ne = t.ne;
    const int64_t e0 = t.e0;
    uint32_t f[kLaneBlocks][kBlock];
#pragma unroll
    for (int q = 0; q < kLaneBlocks; ++q)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int k = 0; k < 4; ++k) f[q][4 * j + k] = nf[q][j][k];
    Blk cb[kLaneBlocks];
#pragma unroll
    for (int q = 0; q < kLaneBlocks; ++q) cb[q] = b[q];

    // A2: hash.  Each block sums pair_term over its 8 pairs (pair index 8 m + i, m the
    // block's index in the path).  Only a path shorter than 16 frames has a block with
    // frames past its end; they read as zero, and a tile without such a block hashes
    // without masks.
    {
      uint32_t z = 0;  // made here: a zero kept across the loop would cost two registers
      asm volatile("" : "+v"(z));
      W.hacc[lane] = ((uint64_t)z << 32) | z;
    }
    wave_sync();
    bool full = true;
#pragma unroll
    for (int q = 0; q < kLaneBlocks; ++q) full &= cb[q].ev < 0 || cb[q].rem == kBlock;
    full = __all(full);
#pragma unroll
    for (int q = 0; q < kLaneBlocks; ++q) {
      if (cb[q].ev >= 0) {
        const uint32_t pb = (uint32_t)(((cb[q].st + kBlock - 1) / kBlock) * (kBlock / 2));
        const uint32_t kx = pb * kPairMulX + kPairAddX, ky = pb * kPairMulY + kPairAddY;
        uint64_t acc = 0;
        if (full) {
#pragma unroll
          for (int i = 0; i < kBlock / 2; ++i) {
            const uint32_t x = f[q][2 * i] + kx + (uint32_t)i * kPairMulX;
            const uint32_t y = f[q][2 * i + 1] + ky + (uint32_t)i * kPairMulY;
            acc += (uint64_t)x * (uint64_t)y;
          }
        } else {
#pragma unroll
          for (int i = 0; i < kBlock / 2; ++i) {
            const uint32_t f0 = 2 * i < cb[q].rem ? f[q][2 * i] : 0u;
            const uint32_t f1 = 2 * i + 1 < cb[q].rem ? f[q][2 * i + 1] : 0u;
            const uint32_t x = f0 + kx + (uint32_t)i * kPairMulX;
            const uint32_t y = f1 + ky + (uint32_t)i * kPairMulY;
            acc += (uint64_t)x * (uint64_t)y;
          }
        }
        atomicAdd((unsigned long long *)&W.hacc[cb[q].ev], (unsigned long long)acc);
      }
    }
    wave_sync();

    // A3: exact dedup.  Lane j resolves event j: a cached resolution of the same hash
    // and length, else the table; every candidate is verified by the event's blocks.
    // (cross-lane reads with every lane active: a disabled source lane reads as zero)
    const int64_t o_end = shfl_i64(o_cur, min(fresh_lane() + 1, 63));
    Probe p{};
    p.state = kResolved;
    // cache entry: claimed (index + kLeader, filled in once resolved) or awaited (index);
    // kFromCache: the current candidate came from the cache; -1: none
    int ce = -1;
    if (lane < ne) {
      p.len = (uint32_t)(o_end - o_cur);
      p.h = finish_hash(W.hacc[lane], (uint64_t)p.len) & a.hash_mask;
      p.slot = (uint32_t)(p.h & a.cap_mask);
      ce = cache_lookup(S, p.h, p.len);
      p.state = ce >= 0 && ce < kLeader ? kWaiting : kProbing;
    }

    for (;;) {
      // a claimed entry is filled in as soon as its path is resolved (or has failed), so
      // lanes waiting on it, in this wave or another, go on
      if (ce >= kLeader && (p.state == kResolved || p.state == kFailed)) {
        cache_fill(S, ce - kLeader, p.len, p.state == kResolved ? p.slot : kNoEntry, p.cbase);
        ce = -1;
      }
      if (p.state == kWaiting) {
        const uint64_t ci = S.cinfo[ce];
        const uint32_t cs = (uint32_t)ci;
        if (cs != kNotReady) {
          if (cs != kNoEntry && (uint32_t)(ci >> 32) == p.len) {
            p.slot = cs;
            p.cbase = S.cbase[ce];
            p.state = p.len == 0 ? kResolved : kCandidate;
            ce = kFromCache;
          } else {
            p.state = kProbing;
            ce = -1;
          }
        }
      }
      if (p.state == kProbing) probe(a, p, e0 + lane, o_cur, (int64_t)p.len);
      if (!__any(p.state == kCandidate)) {
        const bool waiting = __any(p.state == kWaiting);
        if (!waiting && !__any(ce >= kLeader)) break;
        if (waiting) __builtin_amdgcn_s_sleep(1);  // lanes wait on entries other waves resolve
        continue;
      }
      if (lane < ne) {
        uint64_t vp = 0;
        uint32_t lim = 0;
        if (p.state == kCandidate) {
          const uint64_t fi = p.cbase & ~kInStore;
          if (p.cbase & kInStore) {
            vp = (uint64_t)(uintptr_t)(a.pframes + fi);
            lim = (uint32_t)round_store(p.len);
          } else {
            vp = (uint64_t)(uintptr_t)(a.fr + fi);
            const int64_t av = a.n_frames - (int64_t)fi;
            lim = (uint32_t)(av < (int64_t)kWaveFrames ? av : kWaveFrames);
          }
        }
        W.vptr[lane] = vp;
        W.vlim[lane] = lim;
        W.bad[lane] = 0;
      }
      wave_sync();
      // every block of a candidate compares its frames with the candidate's: four
      // 16-byte loads (a block with nothing to verify reads a block of zeros), or, when
      // some block's 16-byte loads would reach past what is readable at its candidate
      // (a candidate at the very end of the batch), 4-byte loads of the path's frames
      {
        uint32_t c[kLaneBlocks][kBlock];
        bool chk[kLaneBlocks];
        gptr cp[kLaneBlocks];
        bool narrow = false;
#pragma unroll
        for (int q = 0; q < kLaneBlocks; ++q) {
          const uint64_t vp = cb[q].ev >= 0 ? W.vptr[cb[q].ev] : 0;
          chk[q] = vp != 0;
          narrow |= chk[q] && (int)W.vlim[cb[q].ev] - cb[q].st < kBlock;
          cp[q] = chk[q] ? (gptr)vp + cb[q].st : (gptr)g_zero_block;
        }
        if (!__any(narrow)) {
#pragma unroll
          for (int q = 0; q < kLaneBlocks; ++q)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const u32x4 v = *(gptr4)(cp[q] + 4 * j);
#pragma unroll
              for (int k = 0; k < 4; ++k) c[q][4 * j + k] = v[k];
            }
        } else {
#pragma unroll
          for (int q = 0; q < kLaneBlocks; ++q)
#pragma unroll
            for (int i = 0; i < kBlock; ++i) c[q][i] = chk[q] && i < cb[q].rem ? cp[q][i] : 0u;
        }
        // frames inside the path must match (in a tile of full blocks, all 16)
#pragma unroll
        for (int q = 0; q < kLaneBlocks; ++q) {
          uint32_t d = 0;
          if (full) {
#pragma unroll
            for (int i = 0; i < kBlock; ++i) d |= c[q][i] ^ f[q][i];
          } else {
#pragma unroll
            for (int i = 0; i < kBlock; ++i) d |= i < cb[q].rem ? c[q][i] ^ f[q][i] : 0u;
          }
          if (chk[q] && d != 0) W.bad[cb[q].ev] = 1;
        }
      }
      wave_sync();
      if (p.state == kCandidate) {
        if (W.bad[lane]) {
          // a table candidate was reached along the probe sequence, so the path is
          // further on; a cached one says nothing about the slots before it
          p.slot = (uint32_t)((ce == kFromCache ? p.h : p.slot + 1) & a.cap_mask);
          p.state = kProbing;
        } else {
          p.state = kResolved;
        }
        if (ce == kFromCache) ce = -1;
      }
      wave_sync();
    }
    // the next tile's frames, and the offsets window after it, are requested only now:
    // vector-memory loads retire in order, so a table or candidate load issued after
    // them would wait for the whole next tile to arrive
    const Tile tn = make_tile(a, W, e_nxt, end, o_nxt, b);
    load_blocks(a, tn, b, nf);
    const int64_t o_nn = tn.kind == kTileFast || tn.kind == kTileSlow ? load_window(a, tn.e0 + tn.ne, end, lane) : 0;
    {
      // buffer store over the tile's entries (the address stays in scalar registers)
      const int64_t eu = uniform64(e0);
      const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
          (void *)(a.slot_of + eu), (short)0, __builtin_amdgcn_readfirstlane(ne * 4), 0x00020000);
      if (lane < ne) __builtin_amdgcn_raw_buffer_store_b32(p.state == kResolved ? p.slot : kNoSlot, r, fresh_lane() * 4, 0, 0);
    }
    o_cur = o_nxt;
    o_nxt = o_nn;
    t = tn;
  }
  // A wave that stopped early (malformed offsets, or a table overflow the host retries)
  // marks the rest of its range unresolved: every entry of slot_of is written once, so
  // the aggregation that follows never reads a stale word as a slot.
  if (t.kind != kTileNone)
    for (int64_t e = t.e0 + lane; e < end; e += 64) a.slot_of[e] = kNoSlot;
}

// Metric sums per slot: one persistent workgroup per CU walks a contiguous event
// range and sums into an LDS map keyed by slot (a hot path costs one map entry per
// workgroup), falling back to HBM atomics when a key's probe window is full.  A key
// already in the map is found with plain LDS reads (broadcast), so hot keys cost no
// atomic compare-and-swap.  Every thread takes kAggUnroll events per round and issues
// all their loads (slot, then the metric row) before touching LDS, so a wave keeps
// kAggUnroll rows in flight.  M is a template parameter: the row is loaded as M
// consecutive 8-byte words, which the compiler merges into wide loads.
//
// The maps are flushed into staging buckets by slot range rather than with one HBM
// atomic per entry and metric (a few million device-scope atomics): a workgroup
// counts its entries per bucket in LDS, reserves room in each bucket with one atomic,
// and writes its entries with plain stores; agg_reduce_kernel then sums every bucket
// in LDS and adds it into delta, each slot owned by one workgroup.
constexpr int kAggThreads = 1024;
constexpr int kAggUnroll = 4;
constexpr int kAggHist = 2048;                            // most buckets a flush can count in LDS
constexpr int kAggLdsBytes = 163840 - kAggHist * 4 - 256;  // map keys and sums
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;
constexpr int kBucketWords = 16384;                        // LDS sums of one bucket (128 KiB)

constexpr int agg_entries(int m) {
  int e = kAggLdsBytes / (4 + 8 * m);
  if (e > 8192) e = 8192;
  return e & ~255;
}
constexpr int agg_bucket_slots(int m) {
  int b = 1;
  while (b * 2 * m <= kBucketWords) b *= 2;
  return b;
}
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

template <int M>
__global__ __launch_bounds__(kAggThreads) void aggregate_kernel(const uint32_t *slot_of, const uint64_t *w, int64_t n,
                                                                uint64_t *delta, AggStage st) {
  constexpr int kEntries = agg_entries(M);
  constexpr int kPer = (kEntries + kAggThreads - 1) / kAggThreads;
  __shared__ uint32_t key[kEntries];
  __shared__ uint64_t sum[kEntries * M];
  __shared__ uint32_t hist[kAggHist];
  const int tid = threadIdx.x;
  for (int i = tid; i < kEntries; i += kAggThreads) key[i] = kEmptyKey;
  for (int i = tid; i < kEntries * M; i += kAggThreads) sum[i] = 0;
  __syncthreads();
  const int64_t b = blockIdx.x, nb = gridDim.x;
  const int64_t lo = b * n / nb, hi = (b + 1) * n / nb;
  for (int64_t e0 = lo + tid; e0 < hi; e0 += (int64_t)kAggThreads * kAggUnroll) {
    uint32_t s[kAggUnroll];
    uint64_t v[kAggUnroll][M];
#pragma unroll
    for (int u = 0; u < kAggUnroll; ++u) {
      const int64_t e = e0 + (int64_t)u * kAggThreads;
      const bool in = e < hi;
      s[u] = in ? slot_of[e] : kNoSlot;
#pragma unroll
      for (int j = 0; j < M; ++j) v[u][j] = in ? w[e * M + j] : 0;
    }
#pragma unroll
    for (int u = 0; u < kAggUnroll; ++u) {
      if (s[u] == kNoSlot) continue;
      uint32_t k = __umulhi(hash32(s[u]), (uint32_t)kEntries);
      int mi = -1;
      for (int t = 0; t < 8; ++t) {
        uint32_t cur = key[k];
        if (cur == kEmptyKey) cur = atomicCAS(&key[k], kEmptyKey, s[u]);
        if (cur == kEmptyKey || cur == s[u]) { mi = (int)k; break; }
        k = k + 1 == (uint32_t)kEntries ? 0 : k + 1;
      }
#pragma unroll
      for (int j = 0; j < M; ++j) {
        if (mi >= 0) atomicAdd((unsigned long long *)&sum[mi * M + j], (unsigned long long)v[u][j]);
        else atomicAdd((unsigned long long *)&delta[(uint64_t)s[u] * M + j], (unsigned long long)v[u][j]);
      }
    }
  }
  __syncthreads();
  const int nbk = (int)st.nbuckets;
  if (nbk == 0 || nbk > kAggHist) {
    for (int k = tid; k < kEntries; k += kAggThreads) {
      const uint32_t sk = key[k];
      if (sk == kEmptyKey) continue;
#pragma unroll
      for (int j = 0; j < M; ++j) {
        const uint64_t v = sum[k * M + j];
        if (v) atomicAdd((unsigned long long *)&delta[(uint64_t)sk * M + j], (unsigned long long)v);
      }
    }
    return;
  }
  // staged flush: rank of every entry within its bucket, then one reservation per bucket
  for (int i = tid; i < nbk; i += kAggThreads) hist[i] = 0;
  __syncthreads();
  uint32_t rank[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int k = tid + j * kAggThreads;
    rank[j] = 0;
    if (k < kEntries && key[k] != kEmptyKey) rank[j] = atomicAdd(&hist[key[k] >> st.bshift], 1u);
  }
  __syncthreads();
  for (int i = tid; i < nbk; i += kAggThreads) {
    const uint32_t c = hist[i];
    hist[i] = c ? atomicAdd(&st.count[i], c) : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int k = tid + j * kAggThreads;
    if (k >= kEntries) continue;
    const uint32_t sk = key[k];
    if (sk == kEmptyKey) continue;
    const uint32_t bk = sk >> st.bshift;
    const uint64_t pos = (uint64_t)hist[bk] + rank[j];
    if (pos < (uint64_t)st.bucket_cap) {
      const uint64_t at = (uint64_t)bk * (uint64_t)st.bucket_cap + pos;
      st.keys[at] = sk;
#pragma unroll
      for (int jj = 0; jj < M; ++jj) st.sums[at * M + jj] = sum[k * M + jj];
    } else {  // the bucket is full (slots far from uniform): add directly
#pragma unroll
      for (int jj = 0; jj < M; ++jj) {
        const uint64_t v = sum[k * M + jj];
        if (v) atomicAdd((unsigned long long *)&delta[(uint64_t)sk * M + jj], (unsigned long long)v);
      }
    }
  }
}

// One workgroup per staging bucket: sum the bucket's entries in LDS, then add them
// into delta (this workgroup is the only writer of the bucket's slots).
template <int M>
__global__ __launch_bounds__(kAggThreads) void agg_reduce_kernel(AggStage st, uint64_t cap, uint64_t *delta) {
  constexpr int kSlots = agg_bucket_slots(M);
  __shared__ uint64_t dense[kSlots * M];
  const int tid = threadIdx.x;
  const uint64_t bk = blockIdx.x;
  for (int i = tid; i < kSlots * M; i += kAggThreads) dense[i] = 0;
  __syncthreads();
  const uint64_t cnt = st.count[bk];
  const uint64_t n = cnt < (uint64_t)st.bucket_cap ? cnt : (uint64_t)st.bucket_cap;
  const uint64_t base = bk * (uint64_t)st.bucket_cap;
  for (uint64_t i = tid; i < n; i += kAggThreads) {
    const uint32_t local = st.keys[base + i] - (uint32_t)(bk << st.bshift);
#pragma unroll
    for (int j = 0; j < M; ++j)
      atomicAdd((unsigned long long *)&dense[local * M + j], (unsigned long long)st.sums[(base + i) * M + j]);
  }
  __syncthreads();
  const uint64_t s0 = bk << st.bshift;
  for (int i = tid; i < kSlots * M; i += kAggThreads) {
    const uint64_t slot = s0 + (uint64_t)(i / M);
    const uint64_t v = dense[i];
    if (slot < cap && v) delta[slot * M + (i % M)] += v;
  }
}

// Slots claimed in this call: a block of 1024 threads scans 4096 slots, counts its
// claims, reserves list positions with one atomic, and writes them (the list order
// is irrelevant: paths get their canonical ids later).  Lengths come from the slot's
// info word; per-block sums of padded and exact lengths go to part[block][2].
constexpr int kCollectThreads = 1024, kCollectPerThread = 4;
__global__ __launch_bounds__(kCollectThreads) void collect_new_kernel(const Slot *slot, uint64_t cap,
                                                                      const int64_t *off, uint32_t *new_slots,
                                                                      int64_t *src_len, uint64_t *padded,
                                                                      unsigned long long *ctr,
                                                                      unsigned long long *part) {
  __shared__ uint32_t cnt;
  __shared__ unsigned long long base, frames, lens;
  if (threadIdx.x == 0) { cnt = 0; frames = 0; lens = 0; }
  __syncthreads();
  uint32_t found[kCollectPerThread], pos[kCollectPerThread];
  int64_t fsrc[kCollectPerThread], flen[kCollectPerThread];
  uint64_t my_frames = 0, my_lens = 0;
  int nf = 0;
  for (int r = 0; r < kCollectPerThread; ++r) {
    const uint64_t s = ((uint64_t)blockIdx.x * kCollectPerThread + r) * kCollectThreads + threadIdx.x;
    if (s >= cap) break;
    const Slot sl = slot[s];
    if (sl.word != kEmptySlot && ((uint32_t)sl.word & kEventRef)) {
      // the claiming event's first frame and length: from info (written right after the
      // claim, so complete once the ingest has finished), else from the offsets
      int64_t src, len;
      if (sl.info != kEmptyInfo && (sl.info & kInfoLongLen) != kInfoLongLen) {
        len = (int64_t)(sl.info & kInfoLongLen);
        src = (int64_t)(sl.info >> 24);
      } else {
        const int64_t e = (int64_t)((uint32_t)sl.word & kRefMask);
        src = off[e];
        len = off[e + 1] - src;
      }
      found[nf] = (uint32_t)s;
      fsrc[nf] = src;
      flen[nf] = len;
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
  for (int i = 0; i < nf; ++i) {
    const uint64_t j = base + pos[i];
    new_slots[j] = found[i];
    src_len[2 * j] = fsrc[i];
    src_len[2 * j + 1] = flen[i];
    padded[j] = (uint64_t)round_store(flen[i]);
  }
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

// Publish the paths first seen in this call: give each a path id, copy its frames into
// the tree's path store (16-frame aligned, zero tail up to its padded length), write its
// checkpoint hashes, its start, length and table slot, and point the slot at the path id
// and the stored frames (the sums are folded in later, by fold_sums_kernel).  Sixteen
// lanes per path, four paths per wave: a lane moves four frames of every 64-frame chunk
// with one 16-byte load (the source, a 4-byte aligned stretch of the batch) and one
// 16-byte store (the store is 64-byte aligned), so a wave has four paths' frames in
// flight.  The chunks of a path up to 128 frames are requested before any is used.  Each
// group of four lanes holds one 16-frame block: the block's frame terms meet by two
// shuffles within the group, and the blocks' prefix sums are carried across chunks.
constexpr int kPublishChunks = 2;  // 64-frame chunks requested ahead
__global__ __launch_bounds__(256) void publish_kernel(PublishArgs a) {
  const int lane = threadIdx.x & 63, g = lane & 15;  // g: lane within the path's 16
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const bool active = i < a.n_new;
  const int64_t src = active ? a.src_len[2 * i] : 0, len = active ? a.src_len[2 * i + 1] : 0;
  const int64_t rl = round_store(len);
  const int64_t start = a.store_used + (active ? (int64_t)a.starts[i] : 0);
  const int64_t full = len / kStoreAlign * kStoreAlign;  // frames of the full blocks
  const int64_t avail = a.n_frames - src;                // frames readable from src
  uint64_t carry = 0;
  u32x4 fq[kPublishChunks];
  for (int64_t k0 = 0; k0 < rl; k0 += 64) {  // uniform within the path's 16 lanes
    const int c = (int)((k0 >> 6) % kPublishChunks);
    if (c == 0) {
#pragma unroll
      for (int u = 0; u < kPublishChunks; ++u) {
        const int64_t k = k0 + 64 * u + 4 * g;  // this lane's first frame of chunk u
        u32x4 v = {0u, 0u, 0u, 0u};
        if (k + 4 <= len && k + 4 <= avail) {
          v = *(gptr4)((gptr)a.fr + src + k);
        } else if (k < len) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = k + e < len ? a.fr[src + k + e] : 0u;
        }
        fq[u] = v;
      }
    }
    u32x4 v = fq[0];
#pragma unroll
    for (int u = 1; u < kPublishChunks; ++u)
      if (c == u) v = fq[u];
    const int64_t k = k0 + 4 * g;
    if (k < rl) *(u32x4 *)(a.pframes + start + k) = v;
    uint64_t t = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) t += k + e < full ? frame_term(v[e], (uint32_t)(k + e)) : 0ull;
    for (int o = 1; o < 4; o <<= 1) {  // the block's sum, on its four lanes
      const uint32_t lo = __shfl_xor((uint32_t)t, o, 64), hi = __shfl_xor((uint32_t)(t >> 32), o, 64);
      t += ((uint64_t)hi << 32) | lo;
    }
    const int base = lane & ~15;  // the path's first lane
    uint64_t bs[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = __shfl((uint32_t)t, base + 4 * q, 64), hi = __shfl((uint32_t)(t >> 32), base + 4 * q, 64);
      bs[q] = ((uint64_t)hi << 32) | lo;
    }
    const int blk = g >> 2;  // this lane's block within the chunk
    uint64_t pre = carry;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q <= blk) pre += bs[q];
    const int64_t b = k0 / kStoreAlign + blk;  // the block within the path
    if ((g & 3) == 3 && (b + 1) * kStoreAlign <= full)
      a.pcp[start / kStoreAlign + b] = finish_hash(pre, (uint64_t)(b + 1) * kStoreAlign) & a.cp_mask;
    carry += bs[0] + bs[1] + bs[2] + bs[3];
  }
  if (active && g == 0) {
    const uint32_t s = a.new_slots[i];
    const int64_t id = a.d_old + i;
    const uint64_t w = a.slot[s].word;
    a.pstart[id] = start;
    a.plen[id] = (uint32_t)len;
    a.pslot[id] = s;
    a.slot[s].word = (w & 0xFFFFFFFF00000000ull) | (uint64_t)id;
    a.slot[s].info = make_info((uint64_t)start, true, (uint64_t)len);
  }
}

// Every path's sums after the batch, into a fresh array (the tree's own sums stay as
// they were until the call commits): paths from earlier calls add their slot's batch
// sums to their old sums, new paths (d >= d_old) take them.
__global__ void fold_sums_kernel(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, const uint64_t *delta,
                                 const uint64_t *old_sums, uint64_t *sums) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= D * m) return;
  const int64_t d = t / m, j = t - d * m;
  const uint64_t x = delta[(uint64_t)pslot[d] * m + j];
  sums[t] = d < d_old ? old_sums[t] + x : x;
}

// Empty the slots published in a call that then failed (they name path ids that the
// tree does not commit).
__global__ void reset_slots_kernel(Slot *slot, const uint32_t *list, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  slot[list[i]].word = kEmptySlot;
  slot[list[i]].info = kEmptyInfo;
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
  uint64_t acc = 0;  // (the stored path is zero-padded to a multiple of 16 frames)
  for (uint32_t p = 0; p < 8 * ((len + 15) / 16); ++p) {
    const int64_t f = st + hash_block_start(p >> 3, len) + 2 * (p & 7);
    acc += pair_term(pframes[f], pframes[f + 1], p);
  }
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
int agg_bucket_shift(int32_t m) {
  switch (m) {
    case 1: return ilog2(agg_bucket_slots(1));
    case 2: return ilog2(agg_bucket_slots(2));
    case 3: return ilog2(agg_bucket_slots(3));
    case 4: return ilog2(agg_bucket_slots(4));
    default: return ilog2(agg_bucket_slots(8));
  }
}
int64_t agg_max_buckets() { return kAggHist; }
int64_t agg_map_entries(int32_t m) {
  switch (m) {
    case 1: return agg_entries(1);
    case 2: return agg_entries(2);
    case 3: return agg_entries(3);
    case 4: return agg_entries(4);
    case 5: return agg_entries(5);
    case 6: return agg_entries(6);
    case 7: return agg_entries(7);
    default: return agg_entries(8);
  }
}
void launch_aggregate(const uint32_t *slot_of, const uint64_t *w, int64_t n, int32_t m, uint64_t *delta,
                      uint64_t cap, int grid, const AggStage &st, hipStream_t s) {
  if (n <= 0) return;
  const bool staged = st.nbuckets > 0 && st.nbuckets <= kAggHist;
  switch (m) {
#define CCT_AGG_CASE(M)                                                                                       \
  case M:                                                                                                     \
    hipLaunchKernelGGL(aggregate_kernel<M>, dim3(grid), dim3(kAggThreads), 0, s, slot_of, w, n, delta, st);  \
    if (staged)                                                                                               \
      hipLaunchKernelGGL(agg_reduce_kernel<M>, dim3((unsigned)st.nbuckets), dim3(kAggThreads), 0, s, st, cap, \
                         delta);                                                                              \
    break;
    CCT_AGG_CASE(1) CCT_AGG_CASE(2) CCT_AGG_CASE(3) CCT_AGG_CASE(4)
    CCT_AGG_CASE(5) CCT_AGG_CASE(6) CCT_AGG_CASE(7) CCT_AGG_CASE(8)
#undef CCT_AGG_CASE
    default: break;
  }
}
int64_t collect_blocks(uint64_t cap) { return (int64_t)((cap + kCollectThreads * kCollectPerThread - 1) /
                                                         (kCollectThreads * kCollectPerThread)); }
void launch_collect_new(const Slot *slot, uint64_t cap, const int64_t *off, uint32_t *new_slots, int64_t *src_len,
                        uint64_t *padded, unsigned long long *ctr, unsigned long long *part, hipStream_t s) {
  const int64_t nb = collect_blocks(cap);
  hipLaunchKernelGGL(collect_new_kernel, dim3((unsigned)nb), dim3(kCollectThreads), 0, s, slot, cap, off, new_slots,
                     src_len, padded, ctr, part);
  hipLaunchKernelGGL(collect_sum_kernel, dim3(1), dim3(256), 0, s, part, nb, ctr);
}
void launch_publish(const PublishArgs &a, hipStream_t s) {
  if (a.n_new <= 0) return;
  hipLaunchKernelGGL(publish_kernel, dim3(blocks_for(a.n_new * 16, 256)), dim3(256), 0, s, a);
}
void launch_fold_sums(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, const uint64_t *delta,
                      const uint64_t *old_sums, uint64_t *sums, hipStream_t s) {
  if (D <= 0) return;
  hipLaunchKernelGGL(fold_sums_kernel, dim3(blocks_for(D * m, 256)), dim3(256), 0, s, D, d_old, m, pslot, delta,
                     old_sums, sums);
}
void launch_reset_slots(Slot *slot, const uint32_t *list, int64_t n, hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(reset_slots_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, slot, list, n);
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
