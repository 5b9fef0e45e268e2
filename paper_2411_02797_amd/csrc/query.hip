// Batched lookup of call paths in a canonical tree: the "query the metric data
// associated with the tree nodes in the matched call paths" step of the analysis API
// (Design, "Performance Analyzer", "Analysis API").
//
// A query path q is a node iff it is a prefix of some distinct full path.  With the
// full paths sorted, the first path p_i >= q is the only candidate that can start
// with q first; if it does, q is node (i, |q|) of p_i's chain, id = base_i + |q| -
// lcp_i - 1 (|q| > lcp_i holds, else p_{i-1} would start with q and be >= q).
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

// record of canonical position i: the path's first frame in the store and its length
__global__ void sorted_paths_kernel(QueryArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.d) return;
  const uint32_t p = a.order[i];
  a.sorted[2 * i] = a.pstart[p];
  a.sorted[2 * i + 1] = a.plen[p];
}

__global__ void query_kernel(QueryArgs a) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= a.q) return;
  const int C = 1 + a.m;
  const int64_t qs = a.qoff[q], qe = a.qoff[q + 1];
  int64_t id = -1;
  if (qs < 0 || qe < qs || qe > a.qn_frames || (q == 0 && qs != 0) || (q + 1 == a.q && qe != a.qn_frames)) {
    atomicOr(a.err, 1ull);
  } else if (qe == qs) {
    id = 0;  // the empty path is the root
  } else {
    const uint32_t *qf = a.qfr + qs;
    const int64_t ql = qe - qs;
    // first i with path_i >= q.  llo and lhi: common prefix of q with the path below the
    // range (path_{lo-1}) and with the path above it (path_hi), 0 for the open ends.  Every
    // path between two paths that share a prefix with q shares it too (paths with a given
    // prefix are consecutive in lexicographic order), so a comparison can skip
    // min(llo, lhi) frames.
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
    if (lo < a.d) {
      l = lhi;  // lo = hi < D: set by the comparison with path_hi, which measured its prefix
      if (l == ql) id = (int64_t)(1 + a.scan_out[lo * C]) + ql - (int64_t)a.lcp[lo] - 1;
      if (id >= a.u || (l == ql && ql <= (int64_t)a.lcp[lo])) {  // cannot happen on a canonical tree
        atomicOr(a.err, 2ull);
        id = -1;
      }
    }
  }
  a.node_ids[q] = id;
  for (int j = 0; j < a.m; ++j) {
    if (a.qexcl) a.qexcl[q * a.m + j] = id >= 0 ? a.excl[id * a.m + j] : 0;
    if (a.qincl) a.qincl[q * a.m + j] = id >= 0 ? a.incl[id * a.m + j] : 0;
  }
}

}  // namespace

void launch_query(const QueryArgs &a, hipStream_t s) {
  if (a.q <= 0) return;
  if (a.d > 0) hipLaunchKernelGGL(sorted_paths_kernel, dim3((unsigned)((a.d + 255) / 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(query_kernel, dim3((unsigned)((a.q + 255) / 256)), dim3(256), 0, s, a);
}

}  // namespace cct
