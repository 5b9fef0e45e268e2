// Per-node statistics beyond the sum.  The paper's tree keeps, for a node's metrics,
// the sum, the minimum, the average and the standard deviation, and a metric recorded at
// the bottom of a call path updates every node along it up to the root (Design,
// "Profiler", "Calling Context Tree").
//
// Kept per distinct path (the tree's path store), folded by every build and merge:
//   count           events on the path
//   min[j]          smallest value of metric j
//   sumsq[j]        sum of squares of metric j, exact modulo 2^128 (two words, low first)
// Per node, on request (cct_stats): the exclusive values are those of the path ending at
// the node; the inclusive ones combine the paths of the node's subtree, which are the
// canonical positions [i, e): i is the path that created the node, e the path that created
// node subend[u] (the first node after the subtree), or D.  Counts and sums of squares come
// from differences of prefix sums over the D paths in canonical order, minima from a
// range-minimum structure over them (in-block prefix and suffix minima over 64-path blocks
// plus a sparse table over the blocks).  The mean is sum / count and the deviation the
// population one, sqrt(n * S2 - S1^2) / n, with the 192-bit integer n * S2 - S1^2 computed
// exactly and rounded once to float64.
#include "common.h"

namespace cct {

namespace {

constexpr uint32_t kStatEmpty = 0xFFFFFFFFu;
constexpr int kStatThreads = 1024;
constexpr int kStatLdsBytes = 163840 - 256;
constexpr int kRmqBlock = 64;  // paths per range-minimum block (one wave)
constexpr int kStageHist = 4096;  // most slot-range buckets of the staged per-slot statistics
constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

constexpr int stat_entries(int m) {
  int e = kStatLdsBytes / (4 + 8 + 24 * m);  // key, count, min and two square words per metric
  if (e > 4096) e = 4096;
  return e & ~63;
}
// the staged map leaves room for the per-bucket counts
constexpr int stat_entries_staged(int m) {
  int e = (kStatLdsBytes - kStageHist * 4 - 64) / (4 + 8 + 24 * m);
  if (e > 4096) e = 4096;
  return e & ~63;
}
// slots per bucket: the largest power of two whose records fit the reduction's LDS
constexpr int kReduceLdsBytes = 120 * 1024;
constexpr int stage_slots(int m) {
  int b = 1;
  while (b * 2 * (1 + 3 * m) * 8 <= kReduceLdsBytes) b *= 2;
  return b;
}

// a += (lo, hi) on two 64-bit words modulo 2^128.  The add that wraps the low word sees
// an old value whose sum with lo overflows, and only that add carries into the high word.
__device__ inline void lds_add_u128(uint64_t *p, uint64_t lo, uint64_t hi) {
  const uint64_t old = atomicAdd((unsigned long long *)p, (unsigned long long)lo);
  const uint64_t h = hi + (old + lo < old ? 1 : 0);
  if (h) atomicAdd((unsigned long long *)(p + 1), (unsigned long long)h);
}
__device__ inline void hbm_add_u128(uint64_t *p, uint64_t lo, uint64_t hi) {
  const uint64_t old = atomicAdd((unsigned long long *)p, (unsigned long long)lo);
  const uint64_t h = hi + (old + lo < old ? 1 : 0);
  if (h) atomicAdd((unsigned long long *)(p + 1), (unsigned long long)h);
}

// The paths new in this batch start from the identity (no sample); the slot -> path map
// inverts pslot for the batch's slots (every event's slot belongs to a path once the new
// paths are published).
__global__ void stats_prepare_kernel(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, uint32_t *path_of_slot,
                                     PathStats p) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= D) return;
  path_of_slot[pslot[i]] = (uint32_t)i;
  if (i < d_old) return;
  p.cnt[i] = 0;
  for (int j = 0; j < m; ++j) {
    p.min[i * m + j] = ~0ull;
    p.sq[(i * m + j) * 2] = 0;
    p.sq[(i * m + j) * 2 + 1] = 0;
  }
}

// One batch's samples, combined per path.  Each workgroup walks a contiguous range of
// events [lo, hi) and combines them in an LDS map keyed by path (hot paths meet there).  An
// event whose key finds no room in its probe window is a miss:
//   staged (kStaged): the miss goes with plain stores to the workgroup's own list (entries
//     lo.. of an N-entry array, so it cannot overflow), and at the end the map's entries go
//     to a second per-workgroup list; both count their entries per path-range bucket, and
//     stats_bucket_kernel and stats_reduce_kernel finish the job without device atomics;
//   otherwise: misses and the map's entries are added into the path arrays with device
//     atomics.
template <int M, bool kStaged>
__global__ __launch_bounds__(kStatThreads) void stats_agg_kernel(const uint32_t *slot_of, const uint32_t *path_of_slot,
                                                                 const uint64_t *w, int64_t n, PathStats ps,
                                                                 StatStage st) {
  constexpr int kE = kStaged ? stat_entries_staged(M) : stat_entries(M);
  constexpr int R = 1 + 3 * M;  // record: count, min[M], sq[M][2]
  __shared__ uint32_t key[kE];
  __shared__ uint64_t cnt[kE];
  __shared__ uint64_t mn[kE * M];
  __shared__ uint64_t sq[kE * M * 2];
  __shared__ uint32_t hist[kStaged ? kStageHist : 1];
  __shared__ uint32_t n_miss, n_map;
  const int tid = threadIdx.x;
  for (int i = tid; i < kE; i += kStatThreads) { key[i] = kStatEmpty; cnt[i] = 0; }
  for (int i = tid; i < kE * M; i += kStatThreads) { mn[i] = ~0ull; sq[2 * i] = 0; sq[2 * i + 1] = 0; }
  if (kStaged) {
    for (int i = tid; i < st.nbuckets; i += kStatThreads) hist[i] = 0;
    if (tid == 0) { n_miss = 0; n_map = 0; }
  }
  __syncthreads();
  const int64_t b = blockIdx.x, nb = gridDim.x;
  const int64_t lo = b * n / nb, hi = (b + 1) * n / nb;
  for (int64_t e = lo + tid; e < hi; e += kStatThreads) {
    const uint32_t slot = slot_of[e];
    uint64_t v[M];
#pragma unroll
    for (int j = 0; j < M; ++j) v[j] = w[e * M + j];
    if (slot == kNoSlot) continue;
    const uint32_t s = path_of_slot[slot];
    uint32_t k = __umulhi(hash32(s), (uint32_t)kE);
    int mi = -1;
    for (int t = 0; t < 8; ++t) {
      uint32_t cur = key[k];
      if (cur == kStatEmpty) cur = atomicCAS(&key[k], kStatEmpty, s);
      if (cur == kStatEmpty || cur == s) { mi = (int)k; break; }
      k = k + 1 == (uint32_t)kE ? 0 : k + 1;
    }
    if (mi >= 0) {
      atomicAdd((unsigned long long *)&cnt[mi], 1ull);
#pragma unroll
      for (int j = 0; j < M; ++j) {
        atomicMin((unsigned long long *)&mn[mi * M + j], (unsigned long long)v[j]);
        lds_add_u128(&sq[(mi * M + j) * 2], v[j] * v[j], __umul64hi(v[j], v[j]));
      }
    } else if (kStaged) {
      const int64_t at = lo + atomicAdd(&n_miss, 1u);
      st.ev_path[at] = s;
#pragma unroll
      for (int j = 0; j < M; ++j) st.ev_w[at * M + j] = v[j];
      atomicAdd(&hist[s >> st.bshift], 1u);
    } else {
      atomicAdd((unsigned long long *)&ps.cnt[s], 1ull);
#pragma unroll
      for (int j = 0; j < M; ++j) {
        atomicMin((unsigned long long *)&ps.min[(uint64_t)s * M + j], (unsigned long long)v[j]);
        hbm_add_u128(&ps.sq[((uint64_t)s * M + j) * 2], v[j] * v[j], __umul64hi(v[j], v[j]));
      }
    }
  }
  __syncthreads();
  if (kStaged) {
    const int64_t nbk = st.nbuckets;
    for (int64_t i = tid; i < nbk; i += kStatThreads) {
      st.hist_ev[i * nb + b] = hist[i];
      hist[i] = 0;
    }
    __syncthreads();
    for (int k = tid; k < kE; k += kStatThreads) {
      const uint32_t s = key[k];
      if (s == kStatEmpty) continue;
      const int64_t at = b * kE + atomicAdd(&n_map, 1u);
      st.map_key[at] = s;
      uint64_t *rec = st.map_rec + at * R;
      rec[0] = cnt[k];
#pragma unroll
      for (int j = 0; j < M; ++j) {
        rec[1 + j] = mn[k * M + j];
        rec[1 + M + 2 * j] = sq[(k * M + j) * 2];
        rec[2 + M + 2 * j] = sq[(k * M + j) * 2 + 1];
      }
      atomicAdd(&hist[s >> st.bshift], 1u);
    }
    __syncthreads();
    for (int64_t i = tid; i < nbk; i += kStatThreads) st.hist_map[i * nb + b] = hist[i];
    if (tid == 0) {
      st.wg_count[2 * b] = n_miss;
      st.wg_count[2 * b + 1] = n_map;
    }
    return;
  }
  for (int k = tid; k < kE; k += kStatThreads) {
    const uint32_t s = key[k];
    if (s == kStatEmpty) continue;
    atomicAdd((unsigned long long *)&ps.cnt[s], (unsigned long long)cnt[k]);
#pragma unroll
    for (int j = 0; j < M; ++j) {
      atomicMin((unsigned long long *)&ps.min[(uint64_t)s * M + j], (unsigned long long)mn[k * M + j]);
      hbm_add_u128(&ps.sq[((uint64_t)s * M + j) * 2], sq[(k * M + j) * 2], sq[(k * M + j) * 2 + 1]);
    }
  }
}

// Workgroup g moves its two lists into their buckets: bucket k's entries from workgroup g
// start at off[k * grid + g] (the exclusive scan of the counts, bucket-major), and a rank
// within them comes from an LDS cursor per bucket.
template <int M>
__global__ __launch_bounds__(kStatThreads) void stats_bucket_kernel(int64_t n, StatStage st) {
  constexpr int R = 1 + 3 * M;
  __shared__ uint64_t cur[kStageHist];
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x, nb = gridDim.x, nbk = st.nbuckets;
  const int64_t lo = b * n / nb;
  for (int64_t i = tid; i < nbk; i += kStatThreads) cur[i] = st.off_ev[i * nb + b];
  __syncthreads();
  const uint32_t n_miss = st.wg_count[2 * b], n_map = st.wg_count[2 * b + 1];
  for (uint32_t i = tid; i < n_miss; i += kStatThreads) {
    const uint32_t s = st.ev_path[lo + i];
    const uint64_t at = atomicAdd((unsigned long long *)&cur[s >> st.bshift], 1ull);
    st.st_ev_path[at] = s;
#pragma unroll
    for (int j = 0; j < M; ++j) st.st_ev_w[at * M + j] = st.ev_w[(lo + i) * M + j];
  }
  __syncthreads();
  for (int64_t i = tid; i < nbk; i += kStatThreads) cur[i] = st.off_map[i * nb + b];
  __syncthreads();
  const int64_t m0 = b * st.map_entries;
  for (uint32_t i = tid; i < n_map; i += kStatThreads) {
    const uint32_t s = st.map_key[m0 + i];
    const uint64_t at = atomicAdd((unsigned long long *)&cur[s >> st.bshift], 1ull);
    st.st_map_key[at] = s;
#pragma unroll
    for (int r = 0; r < R; ++r) st.st_map_rec[at * R + r] = st.map_rec[(m0 + i) * R + r];
  }
}

// One workgroup per bucket of 2^bshift paths: sums its misses and map entries into LDS
// records, then combines them into the paths it owns (no other writer).
template <int M>
__global__ __launch_bounds__(kStatThreads) void stats_reduce_kernel(StatStage st, int64_t D, PathStats ps) {
  constexpr int kB = stage_slots(M), R = 1 + 3 * M;
  __shared__ uint64_t cnt[kB];
  __shared__ uint64_t mn[kB * M];
  __shared__ uint64_t sq[kB * M * 2];
  const int tid = threadIdx.x;
  const int nloc = 1 << st.bshift;
  for (int i = tid; i < nloc; i += kStatThreads) cnt[i] = 0;
  for (int i = tid; i < nloc * M; i += kStatThreads) { mn[i] = ~0ull; sq[2 * i] = 0; sq[2 * i + 1] = 0; }
  __syncthreads();
  const int64_t bk = blockIdx.x, g = st.grid;
  const uint64_t s0 = (uint64_t)bk << st.bshift;
  const uint64_t e0 = st.off_ev[bk * g], e1 = st.off_ev[(bk + 1) * g];
  for (uint64_t i = e0 + tid; i < e1; i += kStatThreads) {
    const uint32_t l = (uint32_t)(st.st_ev_path[i] - s0);
    atomicAdd((unsigned long long *)&cnt[l], 1ull);
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const uint64_t v = st.st_ev_w[i * M + j];
      atomicMin((unsigned long long *)&mn[l * M + j], (unsigned long long)v);
      lds_add_u128(&sq[(l * M + j) * 2], v * v, __umul64hi(v, v));
    }
  }
  const uint64_t m0 = st.off_map[bk * g], m1 = st.off_map[(bk + 1) * g];
  for (uint64_t i = m0 + tid; i < m1; i += kStatThreads) {
    const uint32_t l = (uint32_t)(st.st_map_key[i] - s0);
    const uint64_t *rec = st.st_map_rec + i * R;
    atomicAdd((unsigned long long *)&cnt[l], (unsigned long long)rec[0]);
#pragma unroll
    for (int j = 0; j < M; ++j) {
      atomicMin((unsigned long long *)&mn[l * M + j], (unsigned long long)rec[1 + j]);
      lds_add_u128(&sq[(l * M + j) * 2], rec[1 + M + 2 * j], rec[2 + M + 2 * j]);
    }
  }
  __syncthreads();
  for (int i = tid; i < nloc; i += kStatThreads) {
    const uint64_t path = s0 + (uint64_t)i;
    if ((int64_t)path >= D) break;
    if (!cnt[i]) continue;  // no sample of this path in the batch
    ps.cnt[path] += cnt[i];
#pragma unroll
    for (int j = 0; j < M; ++j) {
      const uint64_t x = mn[i * M + j], old = ps.min[path * M + j];
      ps.min[path * M + j] = x < old ? x : old;
      const uint64_t lo = sq[(i * M + j) * 2], olo = ps.sq[(path * M + j) * 2];
      const uint64_t nlo = olo + lo;
      ps.sq[(path * M + j) * 2] = nlo;
      ps.sq[(path * M + j) * 2 + 1] += sq[(i * M + j) * 2 + 1] + (nlo < olo ? 1 : 0);
    }
  }
}

// ---- node statistics on request ---------------------------------------------------------
// Row of the path at canonical position r for the prefix sums: [count, then per metric the
// four 32-bit limbs of its sum of squares], each in a 64-bit column; a limb column's prefix
// over fewer than 2^32 paths stays below 2^64, so every difference of prefixes is exact.
// cmin[r] holds the path's minima in canonical order.
__global__ void path_rows_kernel(NodeStatArgs a) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a.d) return;
  const uint64_t pid = a.order[r];
  const int C = 1 + 4 * a.m;
  uint64_t *row = a.rows + r * C;
  row[0] = a.pcnt[pid];
  for (int j = 0; j < a.m; ++j) {
    const uint64_t lo = a.psq[(pid * a.m + j) * 2], hi = a.psq[(pid * a.m + j) * 2 + 1];
    row[1 + 4 * j] = lo & 0xFFFFFFFFull;
    row[2 + 4 * j] = lo >> 32;
    row[3 + 4 * j] = hi & 0xFFFFFFFFull;
    row[4 + 4 * j] = hi >> 32;
    a.cmin[r * a.m + j] = a.pmin[pid * a.m + j];
  }
}

// the path at canonical position r created nodes [1 + scan_out[r], 1 + scan_out[r + 1])
// (column 0 of the emission's scan counts new nodes); its last one is where it ends
__global__ void node_path_kernel(NodeStatArgs a) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a.d) return;
  const int C0 = 1 + a.m;
  const uint64_t b = 1 + a.scan_out[r * C0], e = 1 + a.scan_out[(r + 1) * C0];
  for (uint64_t u = b; u < e; ++u) a.node_path[u] = (uint32_t)r;
}

__device__ inline uint64_t min_u64(uint64_t x, uint64_t y) { return x < y ? x : y; }
__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src), hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t shfl_up_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_up((uint32_t)v, o), hi = __shfl_up((uint32_t)(v >> 32), o);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t shfl_down_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_down((uint32_t)v, o), hi = __shfl_down((uint32_t)(v >> 32), o);
  return ((uint64_t)hi << 32) | lo;
}

// one wave per block of kRmqBlock paths: pre[v] = min of the block's paths up to v,
// suf[v] = min from v to the block's end, tab level 0 = the block's minimum
__global__ __launch_bounds__(64) void rmq_block_kernel(NodeStatArgs a) {
  const int64_t blk = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t v = blk * kRmqBlock + lane;
  for (int j = 0; j < a.m; ++j) {
    const uint64_t x = v < a.d ? a.cmin[v * a.m + j] : ~0ull;
    uint64_t p = x, q = x;
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t y = shfl_up_u64(p, o), z = shfl_down_u64(q, o);
      if (lane >= o) p = min_u64(p, y);
      if (lane + o < 64) q = min_u64(q, z);
    }
    if (v < a.d) {
      a.pre[v * a.m + j] = p;
      a.suf[v * a.m + j] = q;
    }
    const uint64_t all = shfl_u64(p, 63);
    if (lane == 0) a.tab[blk * a.m + j] = all;
  }
}

// level k of the sparse table: entry b covers blocks [b, b + 2^k)
__global__ void rmq_level_kernel(NodeStatArgs a, int k) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.nblk) return;
  const int64_t half = (int64_t)1 << (k - 1);
  const int64_t b2 = b + half < a.nblk ? b + half : a.nblk - 1;
  const uint64_t *prev = a.tab + (int64_t)(k - 1) * a.nblk * a.m;
  uint64_t *cur = a.tab + (int64_t)k * a.nblk * a.m;
  for (int j = 0; j < a.m; ++j) cur[b * a.m + j] = min_u64(prev[b * a.m + j], prev[b2 * a.m + j]);
}

__device__ inline int floor_log2_u64(uint64_t x) { return 63 - __clzll((long long)x); }

// minimum of metric j over the paths at canonical positions [l, r] (inclusive, r >= l)
__device__ uint64_t range_min(const NodeStatArgs &a, int64_t l, int64_t r, int j) {
  const int64_t bl = l / kRmqBlock, br = r / kRmqBlock;
  if (bl == br) {
    uint64_t x = ~0ull;
    for (int64_t v = l; v <= r; ++v) x = min_u64(x, a.cmin[v * a.m + j]);
    return x;
  }
  uint64_t x = min_u64(a.suf[l * a.m + j], a.pre[r * a.m + j]);
  if (bl + 1 <= br - 1) {
    const int k = floor_log2_u64((uint64_t)(br - 1 - bl));
    const uint64_t *lev = a.tab + (int64_t)k * a.nblk * a.m;
    x = min_u64(x, min_u64(lev[(bl + 1) * a.m + j], lev[(br - ((int64_t)1 << k)) * a.m + j]));
  }
  return x;
}

// 128-bit value of four limb sums (each below 2^64), modulo 2^128
__device__ inline void limbs_to_u128(uint64_t d0, uint64_t d1, uint64_t d2, uint64_t d3, uint64_t &lo,
                                     uint64_t &hi) {
  lo = d0 + (d1 << 32);
  const uint64_t c = lo < d0 ? 1 : 0;
  hi = (d1 >> 32) + d2 + (d3 << 32) + c;
}

// float64 nearest to the 192-bit integer (w2, w1, w0): the top 64 significant bits with
// every lower bit folded into the lowest one (a sticky bit), converted once, scaled exactly
__device__ inline double u192_to_f64(uint64_t w0, uint64_t w1, uint64_t w2) {
  uint64_t top, rest;
  int e;
  if (w2) {
    const int sh = __clzll((long long)w2);
    top = sh ? (w2 << sh) | (w1 >> (64 - sh)) : w2;
    rest = (sh ? w1 << sh : w1) | w0;
    e = 128 - sh;
  } else if (w1) {
    const int sh = __clzll((long long)w1);
    top = sh ? (w1 << sh) | (w0 >> (64 - sh)) : w1;
    rest = sh ? w0 << sh : w0;
    e = 64 - sh;
  } else {
    return (double)w0;
  }
  return ldexp((double)(top | (rest ? 1ull : 0ull)), e);
}

// population deviation from n, S1 (64-bit) and S2 (128-bit): sqrt(n S2 - S1^2) / n
__device__ inline double deviation(uint64_t n, uint64_t s1, uint64_t s2lo, uint64_t s2hi) {
  if (n == 0) return __longlong_as_double(0x7FF8000000000000ll);
  // n * S2 as three words
  const uint64_t a0 = n * s2lo, a1 = __umul64hi(n, s2lo);
  const uint64_t b0 = n * s2hi, b1 = __umul64hi(n, s2hi);
  const uint64_t w0 = a0, w1 = a1 + b0;
  const uint64_t w2 = b1 + (w1 < a1 ? 1 : 0);
  // minus S1^2
  const uint64_t q0 = s1 * s1, q1 = __umul64hi(s1, s1);
  const uint64_t r0 = w0 - q0, br0 = w0 < q0 ? 1 : 0;
  const uint64_t t1 = w1 - q1, bt = w1 < q1 ? 1 : 0;
  const uint64_t r1 = t1 - br0, br1 = bt | (t1 < br0 ? 1 : 0);
  if (w2 < br1) return __longlong_as_double(0x7FF8000000000000ll);  // negative: a sum wrapped
  const uint64_t r2 = w2 - br1;
  return sqrt(u192_to_f64(r0, r1, r2)) / (double)n;
}

__device__ inline double mean_of(uint64_t s1, uint64_t n) {
  return n ? (double)s1 / (double)n : __longlong_as_double(0x7FF8000000000000ll);
}

__global__ void node_final_kernel(NodeStatArgs a) {
  // one thread per (node, metric): consecutive threads write consecutive output entries
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int m = a.m;
  if (t >= a.u * m) return;
  const int64_t u = t / m;
  const int j = (int)(t - u * m);
  const int C = 1 + 4 * m, C0 = 1 + m;
  // the subtree's paths [i, e) and the path ending at u, if any (the root: all paths, and
  // the empty path if there is one, which sorts first and creates no node)
  int64_t i = 0, e = a.d, own = -1;
  if (u == 0) {
    if (a.d > 0 && a.scan_out[C0] == 0) own = 0;
  } else {
    i = a.node_path[u];
    const uint32_t se = a.subend[u];
    e = se < a.u ? (int64_t)a.node_path[se] : a.d;
    if ((uint64_t)u == a.scan_out[(i + 1) * C0]) own = i;
  }
  const uint64_t *pi = a.prefix + i * C, *pe = a.prefix + e * C, *row = own >= 0 ? a.rows + own * C : nullptr;
  const uint64_t n_ex = row ? row[0] : 0, n_in = pe[0] - pi[0];
  if (j == 0) {
    if (a.out.count_excl) a.out.count_excl[u] = n_ex;
    if (a.out.count_incl) a.out.count_incl[u] = n_in;
  }
  const int64_t o = t;  // u * m + j
  uint64_t ex_lo = 0, ex_hi = 0, in_lo, in_hi;
  if (row) limbs_to_u128(row[1 + 4 * j], row[2 + 4 * j], row[3 + 4 * j], row[4 + 4 * j], ex_lo, ex_hi);
  limbs_to_u128(pe[1 + 4 * j] - pi[1 + 4 * j], pe[2 + 4 * j] - pi[2 + 4 * j], pe[3 + 4 * j] - pi[3 + 4 * j],
                pe[4 + 4 * j] - pi[4 + 4 * j], in_lo, in_hi);
  if (a.out.min_excl) a.out.min_excl[o] = own >= 0 ? a.cmin[own * m + j] : ~0ull;
  if (a.out.min_incl) a.out.min_incl[o] = e > i ? range_min(a, i, e - 1, j) : ~0ull;
  if (a.out.sumsq_excl) { a.out.sumsq_excl[2 * o] = ex_lo; a.out.sumsq_excl[2 * o + 1] = ex_hi; }
  if (a.out.sumsq_incl) { a.out.sumsq_incl[2 * o] = in_lo; a.out.sumsq_incl[2 * o + 1] = in_hi; }
  const uint64_t s_ex = a.excl[o], s_in = a.incl[o];
  if (a.out.mean_excl) a.out.mean_excl[o] = mean_of(s_ex, n_ex);
  if (a.out.mean_incl) a.out.mean_incl[o] = mean_of(s_in, n_in);
  if (a.out.std_excl) a.out.std_excl[o] = deviation(n_ex, s_ex, ex_lo, ex_hi);
  if (a.out.std_incl) a.out.std_incl[o] = deviation(n_in, s_in, in_lo, in_hi);
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

int64_t stats_staged_entries(int32_t m) {
  switch (m) {
    case 1: return stat_entries_staged(1);
    case 2: return stat_entries_staged(2);
    case 3: return stat_entries_staged(3);
    case 4: return stat_entries_staged(4);
    case 5: return stat_entries_staged(5);
    case 6: return stat_entries_staged(6);
    case 7: return stat_entries_staged(7);
    default: return stat_entries_staged(8);
  }
}
int stats_bucket_shift(int32_t m) {
  switch (m) {
    case 1: return ilog2(stage_slots(1));
    case 2: return ilog2(stage_slots(2));
    case 3: return ilog2(stage_slots(3));
    case 4: return ilog2(stage_slots(4));
    case 5: return ilog2(stage_slots(5));
    case 6: return ilog2(stage_slots(6));
    case 7: return ilog2(stage_slots(7));
    default: return ilog2(stage_slots(8));
  }
}
int64_t stats_max_buckets() { return kStageHist; }

void launch_stats_prepare(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, uint32_t *path_of_slot,
                          const PathStats &p, hipStream_t s) {
  if (D > 0)
    hipLaunchKernelGGL(stats_prepare_kernel, dim3(blocks_for(D, 256)), dim3(256), 0, s, D, d_old, m, pslot,
                       path_of_slot, p);
}

// staged (st.nbuckets > 0): the per-path kernel, the scans of its counts, the bucketing and
// the per-bucket reduction; otherwise the per-path kernel with device atomics
void launch_stats_agg(const uint32_t *slot_of, const uint32_t *path_of_slot, const uint64_t *w, int64_t n, int32_t m,
                      int64_t D, int grid, const PathStats &p, const StatStage &st, uint64_t *scan_blk, hipStream_t s) {
  if (n <= 0) return;
  const bool staged = st.nbuckets > 0;
  const int64_t rows = st.nbuckets * grid;
  switch (m) {
#define CCT_STAT_CASE(M)                                                                                        \
  case M:                                                                                                       \
    if (staged) {                                                                                               \
      hipLaunchKernelGGL((stats_agg_kernel<M, true>), dim3(grid), dim3(kStatThreads), 0, s, slot_of,            \
                         path_of_slot, w, n, p, st);                                                            \
      launch_scan(st.hist_ev, rows, 1, scan_blk, st.off_ev, s);                                                \
      launch_scan(st.hist_map, rows, 1, scan_blk, st.off_map, s);                                              \
      hipLaunchKernelGGL(stats_bucket_kernel<M>, dim3(grid), dim3(kStatThreads), 0, s, n, st);                 \
      hipLaunchKernelGGL(stats_reduce_kernel<M>, dim3((unsigned)st.nbuckets), dim3(kStatThreads), 0, s, st, D, \
                         p);                                                                                    \
    } else {                                                                                                    \
      hipLaunchKernelGGL((stats_agg_kernel<M, false>), dim3(grid), dim3(kStatThreads), 0, s, slot_of,           \
                         path_of_slot, w, n, p, st);                                                            \
    }                                                                                                           \
    break;
    CCT_STAT_CASE(1) CCT_STAT_CASE(2) CCT_STAT_CASE(3) CCT_STAT_CASE(4)
    CCT_STAT_CASE(5) CCT_STAT_CASE(6) CCT_STAT_CASE(7) CCT_STAT_CASE(8)
#undef CCT_STAT_CASE
    default: break;
  }
}

int64_t rmq_blocks(int64_t u) { return (u + kRmqBlock - 1) / kRmqBlock; }

void launch_node_stats(const NodeStatArgs &a, uint64_t *scan_blk, hipStream_t s) {
  if (a.d > 0) {
    hipLaunchKernelGGL(path_rows_kernel, dim3(blocks_for(a.d, 256)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(node_path_kernel, dim3(blocks_for(a.d, 256)), dim3(256), 0, s, a);
    hipLaunchKernelGGL(rmq_block_kernel, dim3((unsigned)a.nblk), dim3(64), 0, s, a);
    for (int k = 1; k < a.levels; ++k)
      hipLaunchKernelGGL(rmq_level_kernel, dim3(blocks_for(a.nblk, 256)), dim3(256), 0, s, a, k);
  }
  launch_scan(a.rows, a.d, 1 + 4 * a.m, scan_blk, a.prefix, s);
  hipLaunchKernelGGL(node_final_kernel, dim3(blocks_for(a.u * a.m, 256)), dim3(256), 0, s, a);
}

}  // namespace cct
