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

// compare stored path p with query frames qf[0..ql): sign and common prefix length
__device__ int cmp_path_query(const QueryArgs &a, uint32_t p, const uint32_t *qf, int64_t ql, int64_t *lcp) {
  const int64_t lp = a.plen[p];
  const uint32_t *pf = a.pframes + a.pstart[p];
  const int64_t n = min(lp, ql);
  for (int64_t k = 0; k < n; ++k) {
    const uint32_t x = pf[k], y = qf[k];
    if (x != y) { *lcp = k; return x < y ? -1 : 1; }
  }
  *lcp = n;
  return lp < ql ? -1 : (lp > ql ? 1 : 0);
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
    int64_t lo = 0, hi = a.d;  // first i with path_i >= q
    int64_t l;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (cmp_path_query(a, a.order[mid], qf, ql, &l) < 0) lo = mid + 1; else hi = mid;
    }
    if (lo < a.d) {
      cmp_path_query(a, a.order[lo], qf, ql, &l);
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
  hipLaunchKernelGGL(query_kernel, dim3((unsigned)((a.q + 255) / 256)), dim3(256), 0, s, a);
}

}  // namespace cct
