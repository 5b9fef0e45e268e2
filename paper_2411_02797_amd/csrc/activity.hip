// Correlation-ID join of one flush of GPU activity records with the call paths
// registered at API callbacks.  The profiler emits a unique correlation ID at every
// GPU API callback and associates it with the call path it retrieves there; activity
// records arrive asynchronously and, when the metric buffer is full, are linked to
// their path through that ID and aggregated into the tree (Design, "Profiler", "GPU
// Metrics").
//
// The join runs before the merge and never materializes one path per record:
//   1. corr_range_kernel: the smallest and largest registered ID.  Correlation IDs are
//      normally drawn from a counter, so a flush's IDs span a dense range; when they
//      span less than four entries per registered path, a direct table indexed by
//      ID - min is used (plain stores, one load per lookup), else a hash table;
//   2. corr_insert_kernel: validate the registry's offsets and insert every registered
//      ID: a plain store into the direct table, or a claim in an open-addressing table
//      of 16-byte slots (the 64-bit ID and a 32-bit claim word, registry index + 1,
//      0 = empty: one load reads both);
//   3. corr_unique_kernel: every registered ID must find its own entry (a repeated ID
//      finds the entry of one of its copies only, so repeats are reported whatever the
//      order of the stores was);
//   4. corr_join_kernel: every record looks up its ID; it gets the registry index of
//      its path (or none: counted as unmatched) and stores its own index + 1 into the
//      path's ref word (any record of the path may win: that one owns the path's sums);
//   5. corr_sums_kernel: every owning record stores its metrics as its path's sums and
//      lists the workgroup's other matched records (an LDS counter per workgroup, its
//      own stripe of the list); corr_adds_kernel then adds those records' metrics with
//      atomics (a path is usually named by one record: few atomics, and no zero fill);
//   6. compaction: a scan over (referenced, length) places the referenced paths;
//      compact_meta_kernel writes their batch offsets, source starts and summed metrics,
//      and compact_copy_kernel copies their frames (one thread per 16 batch frames).
//      When every registered path is referenced, the registry itself is the batch and
//      nothing is copied.  The caller merges the batch like any other.
// Merging that batch equals merging one event per matched record with the registered
// path: the tree's sums are additive over events with the same path.
#include <algorithm>

#include "common.h"

namespace cct {

namespace {

// 64-bit finalizer (murmur3 fmix64) spreading correlation IDs over the table
__device__ inline uint64_t corr_hash(uint64_t x) {
  x ^= x >> 33;
  x *= 0xFF51AFD7ED558CCDull;
  x ^= x >> 33;
  x *= 0xC4CEB9FE1A85EC53ull;
  x ^= x >> 33;
  return x;
}

// Registry index of the entry holding `key`, or -1.  Only after every insertion has
// completed (a later kernel): an empty claim word ends the probe sequence.
__device__ inline int64_t corr_find(const ActivityArgs &a, uint64_t key) {
  typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
  uint64_t s = corr_hash(key) & a.cap_mask;
  for (uint64_t step = 0; step <= a.cap_mask; ++step) {
    const u64x2 v = *(const u64x2 *)&a.table[s];  // key and claim word in one load
    const uint32_t c = (uint32_t)v[1];
    if (c == 0) return -1;
    if (v[0] == key) return (int64_t)c - 1;
    s = (s + 1) & a.cap_mask;
  }
  return -1;
}

__device__ inline int64_t dense_find(const ActivityArgs &a, uint64_t key) {
  const uint64_t d = key - a.id_min;  // wraps for key < id_min: out of range
  if (d > a.id_span) return -1;
  const uint32_t c = a.dtab[d];
  return (int64_t)c - 1;
}

__device__ inline int64_t reg_find(const ActivityArgs &a, uint64_t key) {
  return a.dense ? dense_find(a, key) : corr_find(a, key);
}

// min / max of the registered IDs: per workgroup, then one atomic pair per workgroup
constexpr int kRangeThreads = 256;
__global__ __launch_bounds__(kRangeThreads) void corr_range_kernel(ActivityArgs a) {
  __shared__ unsigned long long smin[kRangeThreads / 64], smax[kRangeThreads / 64];
  unsigned long long lo = ~0ull, hi = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.n_reg; i += (int64_t)gridDim.x * blockDim.x) {
    const unsigned long long k = a.reg_corr[i];
    lo = k < lo ? k : lo;
    hi = k > hi ? k : hi;
  }
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long l2 = __shfl_xor(lo, o, 64), h2 = __shfl_xor(hi, o, 64);
    lo = l2 < lo ? l2 : lo;
    hi = h2 > hi ? h2 : hi;
  }
  if ((threadIdx.x & 63) == 0) { smin[threadIdx.x >> 6] = lo; smax[threadIdx.x >> 6] = hi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kRangeThreads / 64; ++w) {
      lo = smin[w] < lo ? smin[w] : lo;
      hi = smax[w] > hi ? smax[w] : hi;
    }
    atomicMin(&a.ctr[kActCtrMin], lo);
    atomicMax(&a.ctr[kActCtrMax], hi);
  }
}

__global__ void corr_insert_kernel(ActivityArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_reg) return;
  const int64_t o0 = a.reg_off[i], o1 = a.reg_off[i + 1];
  bool bad = o0 < 0 || o1 < o0 || o1 > a.reg_n_frames || o1 - o0 > (int64_t)0xFFFFFFFFll;
  if (i == 0) bad |= o0 != 0;
  if (i + 1 == a.n_reg) bad |= o1 != a.reg_n_frames;
  if (bad) atomicOr(&a.ctr[kActCtrError], (unsigned long long)kActBadOffsets);
  const uint64_t key = a.reg_corr[i];
  if (a.dense) {  // key - id_min <= id_span: the range covers every registered ID
    a.dtab[key - a.id_min] = (uint32_t)(i + 1);
    return;
  }
  uint64_t s = corr_hash(key) & a.cap_mask;
  for (uint64_t step = 0; step <= a.cap_mask; ++step) {
    if (atomicCAS(&a.table[s].claim, 0u, (uint32_t)(i + 1)) == 0u) {
      a.table[s].key = key;
      return;
    }
    s = (s + 1) & a.cap_mask;
  }
  atomicOr(&a.ctr[kActCtrError], (unsigned long long)kActTableFull);  // capacity >= 2 entries per ID: unreachable
}

__global__ void corr_unique_kernel(ActivityArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_reg) return;
  if (reg_find(a, a.reg_corr[i]) != i) atomicOr(&a.ctr[kActCtrError], (unsigned long long)kActRepeatedId);
}

// Grid-stride over the records; the unmatched count is summed per workgroup and added
// with one atomic per workgroup (the counter is a single address).
constexpr int kJoinThreads = 256;
__global__ __launch_bounds__(kJoinThreads) void corr_join_kernel(ActivityArgs a) {
  __shared__ unsigned long long wsum[kJoinThreads / 64];
  unsigned long long unmatched = 0;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < a.n_rec; r += (int64_t)gridDim.x * blockDim.x) {
    const int64_t f = reg_find(a, a.rec_corr[r]);
    a.rec_reg[r] = f < 0 ? kNoSlot : (uint32_t)f;
    if (f < 0) ++unmatched;
    else a.ref[f] = (uint32_t)(r + 1);  // the last store names the path's owner
  }
  for (int o = 32; o > 0; o >>= 1) unmatched += __shfl_xor(unmatched, o, 64);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = unmatched;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long t = 0;
    for (int w = 0; w < kJoinThreads / 64; ++w) t += wsum[w];
    if (t) atomicAdd(&a.ctr[kActCtrUnmatched], t);
  }
}

// Sums of each referenced path, first part: the owning record stores its metric row;
// every other matched record is listed in this workgroup's stripe of `list` (stripe b
// starts at b * stride, stride >= the records one workgroup visits), its count in
// cnt[b].
constexpr int kSumThreads = 256;
__global__ __launch_bounds__(kSumThreads) void corr_sums_kernel(ActivityArgs a, const uint64_t *metrics, int32_t m,
                                                                uint64_t *sums, uint32_t *list, int64_t stride,
                                                                uint32_t *cnt) {
  __shared__ uint32_t n;
  if (threadIdx.x == 0) n = 0;
  __syncthreads();
  uint32_t *mine = list + (int64_t)blockIdx.x * stride;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < a.n_rec; r += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t f = a.rec_reg[r];
    if (f == kNoSlot) continue;
    if (a.ref[f] == (uint32_t)(r + 1)) {
      for (int j = 0; j < m; ++j) sums[(int64_t)f * m + j] = metrics[r * m + j];
    } else {
      mine[atomicAdd(&n, 1u)] = (uint32_t)r;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) cnt[blockIdx.x] = n;
}

// Second part (after the first has completed): the listed records add their rows.
__global__ __launch_bounds__(kSumThreads) void corr_adds_kernel(ActivityArgs a, const uint64_t *metrics, int32_t m,
                                                                uint64_t *sums, const uint32_t *list, int64_t stride,
                                                                const uint32_t *cnt) {
  const uint32_t *mine = list + (int64_t)blockIdx.x * stride;
  const uint32_t n = cnt[blockIdx.x];
  for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) {
    const int64_t r = mine[i];
    const int64_t f = a.rec_reg[r];
    for (int j = 0; j < m; ++j)
      atomicAdd((unsigned long long *)&sums[f * m + j], (unsigned long long)metrics[r * m + j]);
  }
}

// Scan input: {referenced, path length if referenced} per registry path.
__global__ void compact_lengths_kernel(ActivityArgs a, uint64_t *rows) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_reg) return;
  const bool used = a.ref[i] != 0;
  rows[2 * i] = used ? 1 : 0;
  rows[2 * i + 1] = used ? (uint64_t)(a.reg_off[i + 1] - a.reg_off[i]) : 0;
}

// Batch entry of every referenced registry path (scan row i: {batch index, first batch
// frame}): its batch offset, where its frames start in the registry, its summed metrics;
// and the batch's final offset (scan row n_reg holds the totals).
__global__ void compact_meta_kernel(ActivityArgs a, const uint64_t *scan, const uint64_t *sums, int32_t m,
                                    int64_t *off_out, int64_t *src_start, uint64_t *met_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) off_out[(int64_t)scan[2 * a.n_reg]] = (int64_t)scan[2 * a.n_reg + 1];  // the batch's end
  if (i >= a.n_reg || a.ref[i] == 0) return;
  const int64_t k = (int64_t)scan[2 * i];
  off_out[k] = (int64_t)scan[2 * i + 1];
  src_start[k] = a.reg_off[i];
  for (int j = 0; j < m; ++j) met_out[k * m + j] = sums[i * m + j];
}

// Frames of the batch, 16 per thread (consecutive threads, consecutive frames): the
// batch path holding the thread's first frame is found by binary search over the batch
// offsets (the last path starting at or before it: empty paths are passed over), then
// the thread walks forward through the paths its frames span.
constexpr int kCopyPerThread = 16;
__global__ void compact_copy_kernel(const int64_t *off, const int64_t *src_start, int64_t n_paths, int64_t n_frames,
                                    const uint32_t *reg_frames, uint32_t *fr_out) {
  const int64_t k0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kCopyPerThread;
  if (k0 >= n_frames) return;
  int64_t lo = 0, hi = n_paths;  // off[lo] <= k0 < off[hi]
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if (off[mid] <= k0) lo = mid;
    else hi = mid;
  }
  int64_t j = lo, end = off[j + 1];
  for (int u = 0; u < kCopyPerThread; ++u) {
    const int64_t k = k0 + u;
    if (k >= n_frames) break;
    while (end <= k) end = off[++j + 1];
    fr_out[k] = reg_frames[src_start[j] + (k - off[j])];
  }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_corr_range(const ActivityArgs &a, hipStream_t s) {
  if (a.n_reg <= 0) return;
  const unsigned grid = (unsigned)std::min<int64_t>(blocks_for(a.n_reg, kRangeThreads), 1024);
  hipLaunchKernelGGL(corr_range_kernel, dim3(grid), dim3(kRangeThreads), 0, s, a);
}

void launch_corr_table(const ActivityArgs &a, hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(corr_insert_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(corr_unique_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a);
}

void launch_corr_join(const ActivityArgs &a, hipStream_t s) {
  if (a.n_rec <= 0) return;
  const unsigned grid = (unsigned)std::min<int64_t>(blocks_for(a.n_rec, kJoinThreads), 2048);
  hipLaunchKernelGGL(corr_join_kernel, dim3(grid), dim3(kJoinThreads), 0, s, a);
}

int64_t corr_sums_grid(int64_t n_rec) { return std::max<int64_t>(1, std::min<int64_t>(blocks_for(n_rec, kSumThreads), 4096)); }

void launch_corr_sums(const ActivityArgs &a, const uint64_t *metrics, int32_t m, uint64_t *sums, uint32_t *list,
                      uint32_t *cnt, hipStream_t s) {
  if (a.n_rec <= 0) return;
  const int64_t grid = corr_sums_grid(a.n_rec);
  // a workgroup visits at most ceil(n_rec / (grid * threads)) records per thread
  const int64_t stride = (a.n_rec + grid * kSumThreads - 1) / (grid * kSumThreads) * kSumThreads;
  hipLaunchKernelGGL(corr_sums_kernel, dim3((unsigned)grid), dim3(kSumThreads), 0, s, a, metrics, m, sums, list,
                     stride, cnt);
  hipLaunchKernelGGL(corr_adds_kernel, dim3((unsigned)grid), dim3(kSumThreads), 0, s, a, metrics, m, sums, list,
                     stride, cnt);
}

void launch_compact_lengths(const ActivityArgs &a, uint64_t *rows, hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(compact_lengths_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a, rows);
}

void launch_compact_gather(const ActivityArgs &a, const uint32_t *reg_frames, const uint64_t *scan,
                           const uint64_t *sums, int32_t m, int64_t n_paths, int64_t n_frames, int64_t *off_out,
                           int64_t *src_start, uint32_t *fr_out, uint64_t *met_out, hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(compact_meta_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a, scan, sums, m, off_out,
                     src_start, met_out);
  if (n_frames > 0)
    hipLaunchKernelGGL(compact_copy_kernel, dim3(blocks_for((n_frames + kCopyPerThread - 1) / kCopyPerThread, 256)),
                       dim3(256), 0, s, off_out, src_start, n_paths, n_frames, reg_frames, fr_out);
}

}  // namespace cct
