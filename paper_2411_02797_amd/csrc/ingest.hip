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
// Layout per workgroup (256 threads, persistent over tiles of consecutive events):
//   - a tile's frames are staged in LDS with 16-byte loads (coalesced HBM stream);
//   - each thread hashes a run of an odd number of consecutive staged frames
//     (odd stride: conflict-free LDS banks) and adds partial sums per event with LDS
//     atomics; the hash is a sum of position-dependent terms, so partial sums over
//     any split of a path combine by addition;
//   - one thread per event probes the table (linear probing, one 64-bit CAS to claim
//     an empty slot); a tag match is verified frame by frame by one wave per event
//     against the candidate's frames (L2/MALL resident: hot paths are few);
//   - metrics go into an LDS map keyed by slot and are flushed to HBM with 64-bit
//     atomics once per workgroup, so a hot path costs one global atomic per
//     workgroup rather than one per event.
#include "common.h"

namespace cct {

namespace {

constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
enum : int32_t { kProbing = 0, kCandidate = 1, kResolved = 2, kFailed = 3 };

struct alignas(16) IngestShared {
  uint32_t fr[kTileFrames + 16];     // staged frames, slot j <-> global frame g0 - lead + j
  uint64_t msum[kMapWords];          // LDS aggregation map sums [entries][m]
  uint32_t mkey[kMapKeys];           // LDS aggregation map keys (table slot ids)
  int64_t off[kTileEvents + 1];      // tile offsets (global)
  uint64_t h[kTileEvents];           // per-event hash accumulator, then final hash
  int64_t repbase[kTileEvents];      // first frame of the candidate's path
  uint32_t probe[kTileEvents];       // current probe slot
  uint32_t steps[kTileEvents];       // slots probed so far (bounded by the capacity)
  int32_t ls[kTileEvents + 1];       // tile-local starts
  int32_t state[kTileEvents];
  int32_t from_store[kTileEvents];   // candidate frames live in the path store
  int32_t mapidx[kTileEvents];
  int32_t flag;
};

__device__ inline int map_entries(int m) {
  int e = kMapWords / m;
  if (e > kMapKeys) e = kMapKeys;
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

// Length of the candidate path referenced by `ref` and where its frames live.
__device__ inline void candidate_frames(const IngestArgs &a, uint32_t ref, int64_t *len, int64_t *base,
                                        int32_t *store) {
  if (ref & kEventRef) {
    int64_t e = ref & kRefMask;
    int64_t s = a.off[e];
    *len = a.off[e + 1] - s;
    *base = s;
    *store = 0;
  } else {
    *len = a.plen[ref];
    *base = a.pstart[ref];
    *store = 1;
  }
}

// Walk the probe sequence of one event until it claims an empty slot (resolved, new
// path) or meets a slot whose tag and length match (candidate, needs verification).
__device__ void probe_event(const IngestArgs &a, IngestShared &S, int i, int64_t ev, int64_t len) {
  const uint64_t h = S.h[i];
  const uint32_t tag = (uint32_t)(h >> 32);
  uint64_t s = S.probe[i];
  for (;;) {
    // every event probes at most `capacity` slots over all its rounds: past the load
    // limit the table may be full, and the event then gives up (overflow)
    if ((uint64_t)S.steps[i]++ > a.cap_mask) {
      atomicOr(&a.ctr[kCtrOverflow], 1ull);
      S.state[i] = kFailed;
      return;
    }
    uint64_t w = __atomic_load_n(&a.slot[s], __ATOMIC_RELAXED);
    if (w == kEmptySlot) {
      const uint64_t mine = ((uint64_t)tag << 32) | (kEventRef | (uint32_t)ev);
      uint64_t prev = atomicCAS((unsigned long long *)&a.slot[s], (unsigned long long)kEmptySlot,
                                (unsigned long long)mine);
      if (prev == kEmptySlot) {
        unsigned long long k = atomicAdd(&a.ctr[kCtrNew], 1ull);
        if (k < a.max_new) {
          a.new_slots[k] = (uint32_t)s;
        } else {
          atomicOr(&a.ctr[kCtrOverflow], 1ull);
        }
        atomicAdd(&a.ctr[kCtrNewFrames], (unsigned long long)len);
        S.probe[i] = (uint32_t)s;
        S.state[i] = kResolved;
        return;
      }
      w = prev;
    }
    if ((uint32_t)(w >> 32) == tag) {
      int64_t clen, cbase;
      int32_t store;
      candidate_frames(a, (uint32_t)w, &clen, &cbase, &store);
      if (clen == len) {
        S.probe[i] = (uint32_t)s;
        if (len == 0) {
          S.state[i] = kResolved;
        } else {
          S.repbase[i] = cbase;
          S.from_store[i] = store;
          S.state[i] = kCandidate;
        }
        return;
      }
    }
    s = (s + 1) & a.cap_mask;
  }
}

// Add one event's metrics into the LDS map (or straight to HBM when the map is full).
__device__ inline int map_insert(IngestShared &S, uint32_t slot, int entries) {
  uint32_t k = hash32(slot) & (uint32_t)(entries - 1);
  for (int t = 0; t < 8; ++t) {
    uint32_t prev = atomicCAS(&S.mkey[k], kEmptyKey, slot);
    if (prev == kEmptyKey || prev == slot) return (int)k;
    k = (k + 1) & (uint32_t)(entries - 1);
  }
  return -1;
}

// Tiles whose frames exceed the LDS staging buffer: one event at a time, the whole
// workgroup striding over its frames in HBM.
__device__ void slow_tile(const IngestArgs &a, IngestShared &S, int64_t e0, int ne, int entries) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = 0; i < ne; ++i) {
    const int64_t gs = S.off[i], len = S.off[i + 1] - gs;
    uint64_t acc = 0;
    for (int64_t k = tid; k < len; k += kIngestThreads) acc += frame_term(a.fr[gs + k], (uint32_t)k);
    acc = wave_sum_u64(acc);
    if (tid == 0) S.h[0] = 0;
    __syncthreads();
    if (lane == 0) atomicAdd((unsigned long long *)&S.h[0], (unsigned long long)acc);
    __syncthreads();
    if (tid == 0) {
      S.h[0] = finish_hash(S.h[0], (uint64_t)len) & a.hash_mask;
      S.probe[0] = (uint32_t)(S.h[0] & a.cap_mask);
      S.steps[0] = 0;
      S.state[0] = kProbing;
    }
    __syncthreads();
    for (;;) {
      if (tid == 0) probe_event(a, S, 0, e0 + i, len);
      __syncthreads();
      if (S.state[0] != kCandidate) break;
      const uint32_t *src = S.from_store[0] ? a.pframes : a.fr;
      const int64_t cb = S.repbase[0];
      bool mism = false;
      for (int64_t k = tid; k < len; k += kIngestThreads) mism |= a.fr[gs + k] != src[cb + k];
      mism = __syncthreads_or(mism);
      if (!mism) {
        if (tid == 0) S.state[0] = kResolved;
        __syncthreads();
        break;
      }
      if (tid == 0) { S.probe[0] = (uint32_t)((S.probe[0] + 1) & a.cap_mask); S.state[0] = kProbing; }
      __syncthreads();
    }
    if (S.state[0] == kResolved) {
      const uint32_t slot = S.probe[0];
      if (tid == 0) S.mapidx[0] = map_insert(S, slot, entries);
      __syncthreads();
      const int mi = S.mapidx[0];
      if (tid < a.m) {
        const uint64_t v = a.w[(e0 + i) * a.m + tid];
        if (mi >= 0) atomicAdd((unsigned long long *)&S.msum[mi * a.m + tid], (unsigned long long)v);
        else atomicAdd((unsigned long long *)&a.delta[(uint64_t)slot * a.m + tid], (unsigned long long)v);
      }
    }
    __syncthreads();
    (void)wave;
  }
}

__global__ __launch_bounds__(kIngestThreads) void ingest_kernel(IngestArgs a) {
  __shared__ IngestShared S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m = a.m;
  const int entries = map_entries(m);
  for (int i = tid; i < kMapKeys; i += kIngestThreads) S.mkey[i] = kEmptyKey;
  for (int i = tid; i < kMapWords; i += kIngestThreads) S.msum[i] = 0;
  __syncthreads();

  for (int64_t tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    if (tid == 0) S.flag = (int)__atomic_load_n(&a.ctr[kCtrOverflow], __ATOMIC_RELAXED);
    __syncthreads();
    if (S.flag) break;
    const int64_t e0 = tile * a.tile_events;
    const int ne = (int)min((int64_t)a.tile_events, a.n_events - e0);

    // A1: offsets of the tile, validated before any frame is read
    for (int i = tid; i <= ne; i += kIngestThreads) S.off[i] = a.off[e0 + i];
    __syncthreads();
    bool bad = false;
    for (int i = tid; i < ne; i += kIngestThreads) bad |= S.off[i + 1] < S.off[i];
    if (tid == 0) {
      bad |= S.off[0] < 0 || S.off[ne] > a.n_frames;
      if (e0 == 0) bad |= S.off[0] != 0;
      if (e0 + ne == a.n_events) bad |= S.off[ne] != a.n_frames;
    }
    if (__syncthreads_or(bad)) {
      if (tid == 0) atomicOr(&a.ctr[kCtrError], (unsigned long long)kErrOffsets);
      continue;
    }
    const int64_t g0 = S.off[0];
    const int64_t span64 = S.off[ne] - g0;
    if (span64 > kTileFrames) {
      slow_tile(a, S, e0, ne, entries);
      continue;
    }
    const int span = (int)span64;
    for (int i = tid; i <= ne; i += kIngestThreads) S.ls[i] = (int32_t)(S.off[i] - g0);
    for (int i = tid; i < ne; i += kIngestThreads) S.h[i] = 0;

    // stage the tile's frames: 16-byte groups aligned in memory and in LDS
    const int lead = (int)(((uintptr_t)a.fr >> 2) + (uint64_t)g0) & 3;
    const uint32_t *gbase = (const uint32_t *)((uintptr_t)a.fr + (uintptr_t)((g0 - lead) * 4));
    const int nq = (lead + span + 3) >> 2;
    for (int q = tid; q < nq; q += kIngestThreads) {
      const int lo = q * 4;
      if (lo >= lead && lo + 4 <= lead + span) {
        const u32x4 v = __builtin_nontemporal_load((const u32x4 *)(gbase + lo));
        *(u32x4 *)&S.fr[lo] = v;
      } else {
        for (int x = 0; x < 4; ++x) {
          const int j = lo + x;
          if (j >= lead && j < lead + span) S.fr[j] = gbase[j];
        }
      }
    }
    __syncthreads();

    // A2: hash.  Thread runs of R (odd) consecutive frames, partial sums per event.
    if (span > 0) {
      const int R = ((span + kIngestThreads - 1) / kIngestThreads) | 1;
      const int p0 = tid * R, p1 = min(span, p0 + R);
      if (p0 < p1) {
        int lo = 0, hi = ne;  // largest i with ls[i] <= p0 (ls[ne] = span > p0)
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (S.ls[mid] <= p0) lo = mid; else hi = mid;
        }
        int cur = lo, cs = S.ls[cur], nx = S.ls[cur + 1];
        uint64_t acc = 0;
        for (int p = p0; p < p1; ++p) {
          if (p >= nx) {
            atomicAdd((unsigned long long *)&S.h[cur], (unsigned long long)acc);
            acc = 0;
            do { ++cur; } while (S.ls[cur + 1] <= p);
            cs = S.ls[cur];
            nx = S.ls[cur + 1];
          }
          acc += frame_term(S.fr[lead + p], (uint32_t)(p - cs));
        }
        atomicAdd((unsigned long long *)&S.h[cur], (unsigned long long)acc);
      }
    }
    __syncthreads();

    // A3: exact dedup.  Probe, verify candidates a wave per event, repeat.
    for (int i = tid; i < ne; i += kIngestThreads) {
      const int64_t len = S.ls[i + 1] - S.ls[i];
      const uint64_t h = finish_hash(S.h[i], (uint64_t)len) & a.hash_mask;
      S.h[i] = h;
      S.probe[i] = (uint32_t)(h & a.cap_mask);
      S.steps[i] = 0;
      S.state[i] = kProbing;
    }
    __syncthreads();
    for (;;) {
      for (int i = tid; i < ne; i += kIngestThreads)
        if (S.state[i] == kProbing) probe_event(a, S, i, e0 + i, S.ls[i + 1] - S.ls[i]);
      __syncthreads();
      bool any = false;
      for (int i = tid; i < ne; i += kIngestThreads) any |= S.state[i] == kCandidate;
      if (!__syncthreads_or(any)) break;
      for (int i = wave; i < ne; i += kIngestThreads / 64) {
        if (S.state[i] != kCandidate) continue;  // uniform across the wave
        const int len = S.ls[i + 1] - S.ls[i];
        const uint32_t *mine = &S.fr[lead + S.ls[i]];
        const uint32_t *src = (S.from_store[i] ? a.pframes : a.fr) + S.repbase[i];
        bool mism = false;
        for (int k = lane; k < len; k += 64) mism |= mine[k] != src[k];
        mism = __any(mism);
        if (lane == 0) {
          if (mism) {
            S.probe[i] = (uint32_t)((S.probe[i] + 1) & a.cap_mask);
            S.state[i] = kProbing;
          } else {
            S.state[i] = kResolved;
          }
        }
      }
      __syncthreads();
    }

    // exclusive aggregation: LDS map keyed by slot, HBM atomics when the map is full
    for (int i = tid; i < ne; i += kIngestThreads)
      S.mapidx[i] = S.state[i] == kResolved ? map_insert(S, S.probe[i], entries) : -2;
    __syncthreads();
    for (int t = tid; t < ne * m; t += kIngestThreads) {
      const int i = t / m, j = t - i * m;
      const int mi = S.mapidx[i];
      if (mi == -2) continue;
      const uint64_t v = a.w[(e0 + i) * m + j];
      if (mi >= 0) atomicAdd((unsigned long long *)&S.msum[mi * m + j], (unsigned long long)v);
      else atomicAdd((unsigned long long *)&a.delta[(uint64_t)S.probe[i] * m + j], (unsigned long long)v);
    }
    __syncthreads();
  }

  // flush the LDS map
  __syncthreads();
  for (int k = tid; k < entries; k += kIngestThreads) {
    const uint32_t key = S.mkey[k];
    if (key == kEmptyKey) continue;
    for (int j = 0; j < m; ++j) {
      const uint64_t v = S.msum[k * m + j];
      if (v) atomicAdd((unsigned long long *)&a.delta[(uint64_t)key * m + j], (unsigned long long)v);
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
  int64_t start = 0;
  if (lane == 0) start = a.store_used + (int64_t)atomicAdd(a.cursor, (unsigned long long)rl);
  start = __shfl(start, 0, 64);
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
