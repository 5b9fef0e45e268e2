// Correlation-ID join of one flush of GPU activity records with the call paths
// registered at API callbacks.  The profiler emits a unique correlation ID at every
// GPU API callback and associates it with the call path it retrieves there; activity
// records arrive asynchronously and, when the metric buffer is full, are linked to
// their path through that ID and aggregated into the tree (Design, "Profiler", "GPU
// Metrics").
//
// The join runs before the merge and never materializes one path per record:
//   1. corr_insert_kernel: validate the registry's offsets and insert every registered
//      ID into an open-addressing table (a 32-bit claim word per slot: registry index
//      + 1, 0 = empty; the 64-bit ID beside it);
//   2. corr_unique_kernel: every registered ID must find its own entry (a repeated ID
//      finds the copy that was inserted first, so repeats are reported whatever the
//      insertion order was);
//   3. corr_join_kernel: every record looks up its ID; it gets the registry index of
//      its path (or none: counted as unmatched), and marks that path as referenced;
//   4. the records' metrics are summed per registry path by the ingest's aggregation
//      kernels (LDS slot maps, staged buckets), keyed by registry index;
//   5. compaction: a scan over (referenced, length) places the referenced paths, and
//      compact_gather_kernel copies their frames and summed metrics into one CSR batch,
//      which the caller merges like any other batch.
// Merging that batch equals merging one event per matched record with the registered
// path: the tree's sums are additive over events with the same path.
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
  uint64_t s = corr_hash(key) & a.cap_mask;
  for (uint64_t step = 0; step <= a.cap_mask; ++step) {
    const uint32_t c = a.claim[s];
    if (c == 0) return -1;
    if (a.keys[s] == key) return (int64_t)c - 1;
    s = (s + 1) & a.cap_mask;
  }
  return -1;
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
  uint64_t s = corr_hash(key) & a.cap_mask;
  for (uint64_t step = 0; step <= a.cap_mask; ++step) {
    if (atomicCAS(&a.claim[s], 0u, (uint32_t)(i + 1)) == 0u) {
      a.keys[s] = key;
      return;
    }
    s = (s + 1) & a.cap_mask;
  }
  atomicOr(&a.ctr[kActCtrError], (unsigned long long)kActTableFull);  // capacity >= 2 entries per ID: unreachable
}

__global__ void corr_unique_kernel(ActivityArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_reg) return;
  if (corr_find(a, a.reg_corr[i]) != i) atomicOr(&a.ctr[kActCtrError], (unsigned long long)kActRepeatedId);
}

__global__ void corr_join_kernel(ActivityArgs a) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool unmatched = false;
  if (r < a.n_rec) {
    const int64_t f = corr_find(a, a.rec_corr[r]);
    unmatched = f < 0;
    a.rec_reg[r] = unmatched ? kNoSlot : (uint32_t)f;
    if (!unmatched) a.ref[f] = 1u;  // every writer stores the same value
  }
  // one atomic per wave for the unmatched count
  const uint64_t bal = __ballot(unmatched);
  if ((threadIdx.x & 63) == 0 && bal) atomicAdd(&a.ctr[kActCtrUnmatched], (unsigned long long)__popcll(bal));
}

// Scan input: {referenced, path length if referenced} per registry path.
__global__ void compact_lengths_kernel(ActivityArgs a, uint64_t *rows) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n_reg) return;
  const bool used = a.ref[i] != 0;
  rows[2 * i] = used ? 1 : 0;
  rows[2 * i + 1] = used ? (uint64_t)(a.reg_off[i + 1] - a.reg_off[i]) : 0;
}

// One wave per registry path: a referenced path is copied to its place in the batch
// (scan row i: {batch index, first frame}), with its summed metrics.
__global__ __launch_bounds__(256) void compact_gather_kernel(ActivityArgs a, const uint32_t *reg_frames,
                                                             const uint64_t *scan, const uint64_t *sums, int32_t m,
                                                             int64_t *off_out, uint32_t *fr_out, uint64_t *met_out) {
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  if (i >= a.n_reg || a.ref[i] == 0) return;
  const int64_t k = (int64_t)scan[2 * i], dst = (int64_t)scan[2 * i + 1];
  const int64_t src = a.reg_off[i], len = a.reg_off[i + 1] - src;
  for (int64_t j = lane; j < len; j += 64) fr_out[dst + j] = reg_frames[src + j];
  if (lane == 0) off_out[k] = dst;
  for (int j = lane; j < m; j += 64) met_out[k * m + j] = sums[i * m + j];
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_corr_table(const ActivityArgs &a, hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(corr_insert_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(corr_unique_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a);
}

void launch_corr_join(const ActivityArgs &a, hipStream_t s) {
  if (a.n_rec <= 0) return;
  hipLaunchKernelGGL(corr_join_kernel, dim3(blocks_for(a.n_rec, 256)), dim3(256), 0, s, a);
}

void launch_compact_lengths(const ActivityArgs &a, uint64_t *rows, hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(compact_lengths_kernel, dim3(blocks_for(a.n_reg, 256)), dim3(256), 0, s, a, rows);
}

void launch_compact_gather(const ActivityArgs &a, const uint32_t *reg_frames, const uint64_t *scan,
                           const uint64_t *sums, int32_t m, int64_t *off_out, uint32_t *fr_out, uint64_t *met_out,
                           hipStream_t s) {
  if (a.n_reg <= 0) return;
  hipLaunchKernelGGL(compact_gather_kernel, dim3(blocks_for(a.n_reg * 64, 256)), dim3(256), 0, s, a, reg_frames,
                     scan, sums, m, off_out, fr_out, met_out);
}

}  // namespace cct
