// Batched lookup of call paths in a canonical tree: the analysis API's step that reads
// the metrics of the tree nodes on the call paths a search matched (Design,
// "Performance Analyzer", "Analysis API").
//
// A query path q is a node iff it is a prefix of some distinct full path.  With the
// full paths sorted, the first path p_i >= q is the only candidate that can start
// with q first; if it does, q is node (i, |q|) of p_i's chain, id = base_i + |q| -
// lcp_i - 1 (|q| > lcp_i holds, else p_{i-1} would start with q and be >= q).
//
// Two ways to find i:
//   - the prefix index (kept with the tree once built): every node (i, l), the depth-l
//     prefix of the path p_i that created it, under a 64-bit hash of that prefix; a query
//     hashes its frames, probes, and verifies every candidate frame by frame against the
//     stored path, so a lookup costs a few round trips;
//   - binary search over the sorted paths (when the index cannot be allocated).
#include "common.h"

namespace cct {

namespace {

// four frames at a 4-byte-aligned address (one 16-byte load)
struct __attribute__((aligned(4))) Frames4 {
  uint32_t f[4];
};

// compare the path at canonical position i with query frames qf[0..ql), both known to
// agree on their first k0 frames: sign and common prefix length.  The path's first frame
// and length come from one 16-byte record; four frames per step, then one at a time.
__device__ int cmp_path_query(const QueryArgs &a, int64_t i, const uint32_t *qf, int64_t ql, int64_t k0,
                              int64_t *lcp) {
  const int64_t *rec = a.sorted + 2 * i;
  const int64_t fs = rec[0], lp = rec[1];
  const uint32_t *pf = a.pframes + fs;
  const int64_t n = min(lp, ql);
  int64_t k = k0;
  for (; k + 4 <= n; k += 4) {
    const Frames4 x = *reinterpret_cast<const Frames4 *>(pf + k);
    const Frames4 y = *reinterpret_cast<const Frames4 *>(qf + k);
    if (x.f[0] != y.f[0] || x.f[1] != y.f[1] || x.f[2] != y.f[2] || x.f[3] != y.f[3]) break;
  }
  for (; k < n; ++k) {
    const uint32_t x = pf[k], y = qf[k];
    if (x != y) { *lcp = k; return x < y ? -1 : 1; }
  }
  *lcp = n;
  return lp < ql ? -1 : (lp > ql ? 1 : 0);
}

// ---- prefix index ----------------------------------------------------------------------
// Hash of a prefix f_0 .. f_{l-1}: the sum of position-dependent terms (a repeated cycle of
// frames does not cancel: both factors move with the position), then a murmur3-style
// finalizer with the length.  Sums extend frame by frame, so one scan along a path gives
// the hash of every prefix.  Correctness never depends on it: every match is verified.
__device__ inline uint64_t prefix_term(uint32_t f, uint32_t k) {
  return (uint64_t)(f + k * 0x9E3779B9u) * (uint64_t)(((f ^ 0x5BD1E995u) + k * 0x85EBCA6Bu) | 1u);
}
__device__ inline uint64_t prefix_key(uint64_t sum, uint64_t len, uint64_t mask) {
  uint64_t h = sum ^ (len * 0xD6E8FEB86659FD93ull);
  h ^= h >> 33;
  h *= 0xFF51AFD7ED558CCDull;
  h ^= h >> 33;
  h *= 0xC4CEB9FE1A85EC53ull;
  h ^= h >> 33;
  return (h & mask) | 1;  // never the empty key 0
}

__device__ inline uint64_t shfl_up_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_up((uint32_t)v, o), hi = __shfl_up((uint32_t)(v >> 32), o);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src), hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}

// One wave per canonical position i: lane k of a 64-frame step holds frame k; an inclusive
// scan of the terms gives the prefix sums; the path's new nodes (depths lcp_i + 1 .. len)
// are inserted by linear probing (a 64-bit CAS claims an empty key; equal keys of other
// nodes just probe on).  The table is at most half full, so every probe sequence ends.
__global__ __launch_bounds__(256) void query_index_kernel(QueryArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  if (i >= a.d) return;
  const int64_t fs = a.sorted[2 * i], len = a.sorted[2 * i + 1];
  const int64_t L = a.lcp[i];
  const uint32_t *pf = a.pframes + fs;
  uint64_t carry = 0;
  for (int64_t k0 = 0; k0 < len; k0 += 64) {
    const int64_t k = k0 + lane;
    const uint64_t t = k < len ? prefix_term(pf[k], (uint32_t)k) : 0;
    uint64_t sc = t;
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t y = shfl_up_u64(sc, o);
      if (lane >= o) sc += y;
    }
    if (k < len && k + 1 > L) {
      const uint64_t key = prefix_key(carry + sc, (uint64_t)(k + 1), a.qhash_mask);
      uint64_t slot = key & a.qcap_mask;
      for (uint64_t probe = 0; probe <= a.qcap_mask; ++probe) {
        const unsigned long long old = atomicCAS((unsigned long long *)&a.qtab[2 * slot], 0ull,
                                                 (unsigned long long)key);
        if (old == 0) {
          a.qtab[2 * slot + 1] = ((uint64_t)(k + 1) << 32) | (uint64_t)i;
          break;
        }
        slot = (slot + 1) & a.qcap_mask;
      }
    }
    carry += shfl_u64(sc, 63);
  }
}

// record of canonical position i: the path's first frame in the store and its length
__global__ void sorted_paths_kernel(QueryArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.d) return;
  const uint32_t p = a.order[i];
  a.sorted[2 * i] = a.pstart[p];
  a.sorted[2 * i + 1] = a.plen[p];
}

// node id of the query through the prefix index, or -1: probe from the query's key; an
// entry with the same key and length is checked frame by frame against its path
__device__ int64_t index_lookup(const QueryArgs &a, const uint32_t *qf, int64_t ql) {
  const int C = 1 + a.m;
  uint64_t sum = 0;
  int64_t k = 0;
  for (; k + 4 <= ql; k += 4) {
    const Frames4 x = *reinterpret_cast<const Frames4 *>(qf + k);
#pragma unroll
    for (int j = 0; j < 4; ++j) sum += prefix_term(x.f[j], (uint32_t)(k + j));
  }
  for (; k < ql; ++k) sum += prefix_term(qf[k], (uint32_t)k);
  const uint64_t key = prefix_key(sum, (uint64_t)ql, a.qhash_mask);
  uint64_t slot = key & a.qcap_mask;
  for (uint64_t probe = 0; probe <= a.qcap_mask; ++probe) {
    const uint64_t kk = a.qtab[2 * slot];
    if (kk == 0) return -1;  // an empty slot ends the probe sequence
    if (kk == key) {
      const uint64_t v = a.qtab[2 * slot + 1];
      const int64_t i = (int64_t)(uint32_t)v, l = (int64_t)(v >> 32);
      int64_t common;
      if (l == ql && cmp_path_query(a, i, qf, ql, 0, &common) >= 0 && common == ql) {
        const int64_t id = (int64_t)(1 + a.scan_out[i * C]) + ql - (int64_t)a.lcp[i] - 1;
        if (id >= a.u || ql <= (int64_t)a.lcp[i]) {  // cannot happen on a canonical tree
          atomicOr(a.err, 2ull);
          return -1;
        }
        return id;
      }
    }
    slot = (slot + 1) & a.qcap_mask;
  }
  return -1;
}

// node id of the query by binary search over the sorted paths, or -1: the first i with
// path_i >= q.  llo and lhi: common prefix of q with the path below the range (path_{lo-1})
// and with the path above it (path_hi), 0 for the open ends.  Every path between two paths
// that share a prefix with q shares it too (paths with a given prefix are consecutive in
// lexicographic order), so a comparison can skip min(llo, lhi) frames.
__device__ int64_t search_lookup(const QueryArgs &a, const uint32_t *qf, int64_t ql) {
  const int C = 1 + a.m;
  int64_t lo = 0, hi = a.d, llo = 0, lhi = 0;
  int64_t l;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (cmp_path_query(a, mid, qf, ql, min(llo, lhi), &l) < 0) {
      lo = mid + 1;
      llo = l;
    } else {
      hi = mid;
      lhi = l;
    }
  }
  int64_t id = -1;
  if (lo < a.d) {
    l = lhi;  // lo = hi < D: set by the comparison with path_hi, which measured its prefix
    if (l == ql) id = (int64_t)(1 + a.scan_out[lo * C]) + ql - (int64_t)a.lcp[lo] - 1;
    if (id >= a.u || (l == ql && ql <= (int64_t)a.lcp[lo])) {  // cannot happen on a canonical tree
      atomicOr(a.err, 2ull);
      id = -1;
    }
  }
  return id;
}

// The query batch's offsets, checked before any output is written: err bit 0 when they
// do not start at 0, decrease, leave the frames or do not end at n_frames.
__global__ void query_check_kernel(QueryArgs a) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.q) return;
  const int64_t qs = a.qoff[q], qe = a.qoff[q + 1];
  if (qs < 0 || qe < qs || qe > a.qn_frames || (q == 0 && qs != 0) || (q + 1 == a.q && qe != a.qn_frames))
    atomicOr(a.err, 1ull);
}

__global__ void query_kernel(QueryArgs a) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.q) return;
  const int64_t qs = a.qoff[q], qe = a.qoff[q + 1];
  int64_t id = -1;
  if (qs < 0 || qe < qs || qe > a.qn_frames || (q == 0 && qs != 0) || (q + 1 == a.q && qe != a.qn_frames)) {
    atomicOr(a.err, 1ull);
  } else if (qe == qs) {
    id = 0;  // the empty path is the root
  } else if (a.qtab) {
    id = index_lookup(a, a.qfr + qs, qe - qs);
  } else {
    id = search_lookup(a, a.qfr + qs, qe - qs);
  }
  a.node_ids[q] = id;
  for (int j = 0; j < a.m; ++j) {
    if (a.qexcl) a.qexcl[q * a.m + j] = id >= 0 ? a.excl[id * a.m + j] : 0;
    if (a.qincl) a.qincl[q * a.m + j] = id >= 0 ? a.incl[id * a.m + j] : 0;
  }
}

}  // namespace

void launch_sorted_paths(const QueryArgs &a, hipStream_t s) {
  if (a.d > 0) hipLaunchKernelGGL(sorted_paths_kernel, dim3((unsigned)((a.d + 255) / 256)), dim3(256), 0, s, a);
}

void launch_query_index(const QueryArgs &a, hipStream_t s) {
  if (a.d > 0) hipLaunchKernelGGL(query_index_kernel, dim3((unsigned)((a.d * 64 + 255) / 256)), dim3(256), 0, s, a);
}

void launch_query_check(const QueryArgs &a, hipStream_t s) {
  if (a.q > 0) hipLaunchKernelGGL(query_check_kernel, dim3((unsigned)((a.q + 255) / 256)), dim3(256), 0, s, a);
}

void launch_query(const QueryArgs &a, hipStream_t s) {
  if (a.q > 0) hipLaunchKernelGGL(query_kernel, dim3((unsigned)((a.q + 255) / 256)), dim3(256), 0, s, a);
}

}  // namespace cct
