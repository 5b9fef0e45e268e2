// Bottom-up view of the tree: the metrics of every frame aggregated over all the call
// paths it appears on.  The flame-graph view of the paper offers a top-down view (the
// tree itself) and a bottom-up view that aggregates the metrics of the same node across
// different call paths (Implementation, "GUI", "Flame Graph Visualization").
//
// For a frame f:
//   excl(f) = sum over the nodes labelled f of their exclusive sums (the events whose
//             path ends with f);
//   incl(f) = sum over the events whose path contains f, each counted once however often
//             f recurs on its path = sum of the inclusive sums of the topmost nodes
//             labelled f (no proper ancestor labelled f): every such event passes through
//             exactly one of them.
//
// On the canonical tree (preorder ids, subtree of u = ids [u, subend[u])):
//   1. the nodes 1 .. U-1 are sorted by frame with a stable radix sort (four passes of 8
//      bits), so each frame's nodes form a group in preorder;
//   2. a node is topmost iff no earlier node of its group has a subtree that reaches past
//      it: one exclusive max-scan over (group index << 32 | subend) decides every node
//      (an earlier group has a smaller high word);
//   3. every node learns its group (scattered back to node order), and the aggregation
//      kernels of the ingest (LDS maps per workgroup, staged buckets) sum the nodes'
//      exclusive sums, and the topmost nodes' inclusive sums, per group: the sums are read
//      in node order, and hot frames meet in LDS.
#include <algorithm>

#include "common.h"

namespace cct {

namespace {

// ---- stable LSD radix sort of (uint32 key, uint32 value) pairs ---------------------------
constexpr int kRsThreads = 256, kRsPerThread = 8, kRsTile = kRsThreads * kRsPerThread;

// digit histogram of one tile, stored digit-major: hist[digit * nblk + block]
__global__ __launch_bounds__(kRsThreads) void rs_hist_kernel(const uint32_t *keys, int64_t n, int shift, int64_t nblk,
                                                            uint64_t *hist) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t t0 = (int64_t)blockIdx.x * kRsTile;
  for (int k = 0; k < kRsPerThread; ++k) {
    const int64_t i = t0 + (int64_t)k * kRsThreads + threadIdx.x;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

// Scatter of one tile to its digits' places (offs: exclusive scan of the digit-major
// histogram).  The tile is read in rounds of 256 consecutive elements; within a round an
// element's rank among equal digits comes from its wave (8 ballots find the lanes with
// the same digit) and the counts of the waves before it, so equal keys keep their order.
__global__ __launch_bounds__(kRsThreads) void rs_scatter_kernel(const uint32_t *keys, const uint32_t *vals, int64_t n,
                                                               int shift, int64_t nblk, const uint64_t *offs,
                                                               uint32_t *keys_out, uint32_t *vals_out) {
  constexpr int kW = kRsThreads / 64;
  __shared__ uint32_t base[256];
  __shared__ uint32_t cnt[kW][256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  base[tid] = (uint32_t)offs[(int64_t)tid * nblk + blockIdx.x];
  for (int w = 0; w < kW; ++w) cnt[w][tid] = 0;
  __syncthreads();
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int64_t t0 = (int64_t)blockIdx.x * kRsTile;
  for (int k = 0; k < kRsPerThread; ++k) {
    const int64_t i = t0 + (int64_t)k * kRsThreads + tid;
    const bool valid = i < n;
    const uint32_t key = valid ? keys[i] : 0u, val = valid ? vals[i] : 0u;
    const uint32_t d = (key >> shift) & 255u;
    uint64_t same = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t ones = __ballot((d >> b) & 1u);
      same &= ((d >> b) & 1u) ? ones : ~ones;
    }
    const uint32_t rank = (uint32_t)__popcll(same & below);
    if (valid && rank == 0) cnt[wave][d] = (uint32_t)__popcll(same);
    __syncthreads();
    if (valid) {
      uint32_t pos = base[d] + rank;
      for (int w = 0; w < wave; ++w) pos += cnt[w][d];
      keys_out[pos] = key;
      vals_out[pos] = val;
    }
    __syncthreads();
    uint32_t add = 0;
    for (int w = 0; w < kW; ++w) {
      add += cnt[w][tid];
      cnt[w][tid] = 0;
    }
    base[tid] += add;
    __syncthreads();
  }
}

// ---- exclusive max-scan of uint64 (identity 0) -------------------------------------------
constexpr int kMsThreads = 256, kMsPer = 4, kMsRows = kMsThreads * kMsPer;

__device__ inline uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ inline uint64_t xor_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_xor((uint32_t)v, o, 64), hi = __shfl_xor((uint32_t)(v >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t up_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_up((uint32_t)v, o, 64), hi = __shfl_up((uint32_t)(v >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}

__global__ __launch_bounds__(kMsThreads) void ms_reduce_kernel(const uint64_t *in, int64_t n, uint64_t *blk) {
  __shared__ uint64_t part[kMsThreads / 64];
  const int64_t r0 = (int64_t)blockIdx.x * kMsRows;
  uint64_t m = 0;
  for (int k = 0; k < kMsPer; ++k) {
    const int64_t r = r0 + (int64_t)k * kMsThreads + threadIdx.x;
    if (r < n) m = umax64(m, in[r]);
  }
  for (int o = 32; o > 0; o >>= 1) m = umax64(m, xor_u64(m, o));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kMsThreads / 64; ++w) m = umax64(m, part[w]);
    blk[blockIdx.x] = umax64(part[0], m);
  }
}

// exclusive max-scan of the block maxima in place (one workgroup)
__global__ __launch_bounds__(kMsThreads) void ms_blocks_kernel(uint64_t *blk, int64_t nblk) {
  __shared__ uint64_t part[kMsThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t carry = 0;
  for (int64_t b0 = 0; b0 < nblk; b0 += kMsThreads) {
    const int64_t b = b0 + tid;
    const uint64_t v = b < nblk ? blk[b] : 0;
    uint64_t x = v;  // inclusive within the wave
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t y = up_u64(x, o);
      if (lane >= o) x = umax64(x, y);
    }
    if (lane == 63) part[wave] = x;
    __syncthreads();
    uint64_t before = carry;
    for (int w = 0; w < wave; ++w) before = umax64(before, part[w]);
    const uint64_t prev = up_u64(x, 1);  // every lane takes part in the shuffle
    const uint64_t excl = lane ? umax64(before, prev) : before;
    uint64_t tot = carry;
    for (int w = 0; w < kMsThreads / 64; ++w) tot = umax64(tot, part[w]);
    __syncthreads();
    if (b < nblk) blk[b] = excl;
    carry = tot;
  }
}

__global__ __launch_bounds__(kMsThreads) void ms_final_kernel(const uint64_t *in, int64_t n, const uint64_t *blk,
                                                             uint64_t *out) {
  __shared__ uint64_t part[kMsThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kMsRows + (int64_t)tid * kMsPer;  // kMsPer consecutive rows
  uint64_t v[kMsPer], m = 0;
  for (int k = 0; k < kMsPer; ++k) {
    v[k] = r0 + k < n ? in[r0 + k] : 0;
    m = umax64(m, v[k]);
  }
  uint64_t x = m;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = up_u64(x, o);
    if (lane >= o) x = umax64(x, y);
  }
  if (lane == 63) part[wave] = x;
  __syncthreads();
  uint64_t run = blk[blockIdx.x];
  for (int w = 0; w < wave; ++w) run = umax64(run, part[w]);
  const uint64_t prev = up_u64(x, 1);  // every lane takes part in the shuffle
  if (lane) run = umax64(run, prev);
  for (int k = 0; k < kMsPer; ++k) {
    if (r0 + k < n) out[r0 + k] = run;
    run = umax64(run, v[k]);
  }
}

// ---- the view -----------------------------------------------------------------------------
__global__ void bu_keys_kernel(const uint32_t *frame, int64_t n, uint32_t *keys, uint32_t *vals) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  keys[i] = frame[i + 1];
  vals[i] = (uint32_t)(i + 1);
}

__global__ void bu_heads_kernel(const uint32_t *K, int64_t n, uint64_t *head) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  head[i] = (i == 0 || K[i] != K[i - 1]) ? 1 : 0;
}

// tag of sorted position i: (group << 32) | subend of its node; group = inclusive count of
// heads - 1.  Group starts are recorded for the output (gstart[G] = n).
__global__ void bu_tag_kernel(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint32_t *subend,
                              int64_t n, uint64_t *tag, int64_t *gstart) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint64_t g = gscan[i] + head[i] - 1;
  tag[i] = (g << 32) | subend[V[i]];
  if (head[i]) gstart[g] = i;
  if (i == n - 1) gstart[g + 1] = n;  // g + 1 = the number of groups
}

// group of every node in node order: slot_ex[v] = group of v, slot_in[v] = group of v if
// v is the topmost node of its frame on its root path, else none; the root is in no group
__global__ void bu_slots_kernel(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint64_t *mx,
                                int64_t n, uint32_t *slot_ex, uint32_t *slot_in) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) slot_ex[0] = slot_in[0] = kNoSlot;
  if (i >= n) return;
  const uint64_t g = gscan[i] + head[i] - 1;
  const uint32_t v = V[i];
  const bool top = (mx[i] >> 32) != g || (uint64_t)v >= (mx[i] & 0xFFFFFFFFull);
  slot_ex[v] = (uint32_t)g;
  slot_in[v] = top ? (uint32_t)g : kNoSlot;
}

// frame of every group (its first sorted position)
__global__ void bu_frames_kernel(const uint32_t *K, const int64_t *gstart, int64_t G, uint32_t *frames) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g < G) frames[g] = K[gstart[g]];
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

int64_t radix_blocks(int64_t n) { return (n + kRsTile - 1) / kRsTile; }
int64_t maxscan_blocks(int64_t n) { return (n + kMsRows - 1) / kMsRows; }

void launch_radix_sort(uint32_t *keys, uint32_t *vals, uint32_t *keys_tmp, uint32_t *vals_tmp, int64_t n,
                       uint64_t *hist, uint64_t *offs, uint64_t *scan_blk, hipStream_t s) {
  if (n <= 0) return;
  const int64_t nblk = radix_blocks(n);
  uint32_t *ki = keys, *vi = vals, *ko = keys_tmp, *vo = vals_tmp;
  for (int shift = 0; shift < 32; shift += 8) {
    hipLaunchKernelGGL(rs_hist_kernel, dim3((unsigned)nblk), dim3(kRsThreads), 0, s, ki, n, shift, nblk, hist);
    launch_scan(hist, 256 * nblk, 1, scan_blk, offs, s);
    hipLaunchKernelGGL(rs_scatter_kernel, dim3((unsigned)nblk), dim3(kRsThreads), 0, s, ki, vi, n, shift, nblk, offs,
                       ko, vo);
    uint32_t *t = ki; ki = ko; ko = t;
    t = vi; vi = vo; vo = t;
  }
  // four passes: the result is back in keys / vals
}

void launch_maxscan(const uint64_t *in, int64_t n, uint64_t *blk, uint64_t *out, hipStream_t s) {
  if (n <= 0) return;
  const int64_t nblk = maxscan_blocks(n);
  hipLaunchKernelGGL(ms_reduce_kernel, dim3((unsigned)nblk), dim3(kMsThreads), 0, s, in, n, blk);
  hipLaunchKernelGGL(ms_blocks_kernel, dim3(1), dim3(kMsThreads), 0, s, blk, nblk);
  hipLaunchKernelGGL(ms_final_kernel, dim3((unsigned)nblk), dim3(kMsThreads), 0, s, in, n, blk, out);
}

void launch_bu_keys(const uint32_t *frame, int64_t n, uint32_t *keys, uint32_t *vals, hipStream_t s) {
  if (n > 0) hipLaunchKernelGGL(bu_keys_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, frame, n, keys, vals);
}
void launch_bu_heads(const uint32_t *K, int64_t n, uint64_t *head, hipStream_t s) {
  if (n > 0) hipLaunchKernelGGL(bu_heads_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, K, n, head);
}
void launch_bu_tag(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint32_t *subend, int64_t n,
                   uint64_t *tag, int64_t *gstart, hipStream_t s) {
  if (n > 0)
    hipLaunchKernelGGL(bu_tag_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, V, head, gscan, subend, n, tag, gstart);
}
void launch_bu_slots(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint64_t *mx, int64_t n,
                     uint32_t *slot_ex, uint32_t *slot_in, hipStream_t s) {
  hipLaunchKernelGGL(bu_slots_kernel, dim3(blocks_for(std::max<int64_t>(n, 1), 256)), dim3(256), 0, s, V, head, gscan,
                     mx, n, slot_ex, slot_in);
}
void launch_bu_frames(const uint32_t *K, const int64_t *gstart, int64_t G, uint32_t *frames, hipStream_t s) {
  if (G > 0) hipLaunchKernelGGL(bu_frames_kernel, dim3(blocks_for(G, 256)), dim3(256), 0, s, K, gstart, G, frames);
}

}  // namespace cct
