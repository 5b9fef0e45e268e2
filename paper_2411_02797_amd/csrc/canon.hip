// Canonical tree from the D distinct full paths (path store + exclusive sums).
//
// The paper's tree is a pointer structure with no node numbering (Design,
// "Profiler", "Calling Context Tree"); this library numbers nodes by the unsigned
// lexicographic rank of their root path.  With the D distinct full paths sorted
// lexicographically (p_0 < p_1 < ...) and lcp_i the length of the longest common
// prefix of p_{i-1} and p_i (lcp_0 = 0):
//   - path i contributes exactly the nodes p_i[0..l) for l in (lcp_i, len_i] (its
//     chain), which are new and, in id order, follow every node of the earlier
//     paths; so node ids are base_i + (l - lcp_i - 1) with base_i = 1 + sum of the
//     chain lengths (len - lcp) of earlier paths, and U = 1 + sum of all of them;
//   - the parent of a chain's first node is the node p_i[0..lcp_i), created by the
//     largest c < i with lcp_c < lcp_i (previous smaller value); every other chain
//     node's parent is the node before it;
//   - the paths through node (i, l) are exactly p_i .. p_{e-1}, e the first j > i
//     with lcp_j < l (next smaller value), and since a metric is added at the last
//     node of its path and then counted at every node up to the root (Design,
//     "Profiler", "Calling Context Tree"), inclusive(i, l) = S[e] - S[i] with S the
//     exclusive prefix sum of the per-path sums in sorted order (mod 2^64);
//   - exclusive(i, len_i) = the sums of path i, every other node has none (the empty
//     path, which sorts first, puts its sums on the root).
// Every step is a sort, a scan or an O(log D) search: the number of kernel launches
// does not grow with the tree depth.
#include <algorithm>

#include "common.h"

namespace cct {

namespace {

constexpr uint32_t kInf = 0xFFFFFFFFu;
constexpr int kSortBlock = 1024;   // keys per block-local bitonic sort
constexpr int kMergeItems = 8;     // outputs per thread per merge pass
constexpr int kScanRows = 1024;    // rows per scan block

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline u32x4 ld4(const uint32_t *p) { return *(const u32x4 *)p; }

// Exact comparison of two stored paths: returns <0, 0, >0 and their lcp.  Starts are
// 16-frame aligned and tails are padded, so 16-byte loads never leave a path's slot.
__device__ int path_cmp_exact(const CanonArgs &a, uint32_t x, uint32_t y, uint32_t from, uint32_t *lcp) {
  const uint32_t lx = a.plen[x], ly = a.plen[y];
  const uint32_t *px = a.pframes + a.pstart[x], *py = a.pframes + a.pstart[y];
  const uint32_t n = min(lx, ly);
  for (uint32_t q = from & ~15u; q < n; q += 16) {
    u32x4 vx[4], vy[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) { vx[c] = ld4(px + q + 4 * c); vy[c] = ld4(py + q + 4 * c); }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t k = q + 4 * c + e;
        if (k < n && vx[c][e] != vy[c][e]) {
          *lcp = k;
          return vx[c][e] < vy[c][e] ? -1 : 1;
        }
      }
    }
  }
  *lcp = n;
  return lx < ly ? -1 : (lx > ly ? 1 : 0);
}

// Comparison accelerated by checkpoint hashes (prefix hashes every 16 frames): skip
// to the first 16-frame block whose prefix hashes differ, then compare frames
// there.  A hash collision can only make this answer wrong, never loop or fault;
// the exact verification after the sort catches any resulting misorder.
__device__ bool path_less(const CanonArgs &a, uint32_t x, uint32_t y) {
  if (x == kInf) return false;
  if (y == kInf) return true;
  uint32_t l;
  if (a.exact) return path_cmp_exact(a, x, y, 0, &l) < 0;
  const uint32_t lx = a.plen[x], ly = a.plen[y];
  const int64_t sx = a.pstart[x], sy = a.pstart[y];
  const uint32_t n = min(lx, ly), nb = n / kStoreAlign;
  const uint64_t *cx = a.pcp + sx / kStoreAlign, *cy = a.pcp + sy / kStoreAlign;
  uint32_t b = 0;
  for (; b + 4 <= nb; b += 4) {
    uint64_t hx[4], hy[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) { hx[c] = cx[b + c]; hy[c] = cy[b + c]; }
    int c = 0;
    while (c < 4 && hx[c] == hy[c]) ++c;
    if (c < 4) { b += c; goto found; }
  }
  for (; b < nb; ++b)
    if (cx[b] != cy[b]) break;
found:
  {
    // first differing frame is in block b (or in the partial block past nb)
    const int r = path_cmp_exact(a, x, y, b * kStoreAlign, &l);
    if (l < min(n, (b + 1) * kStoreAlign) || b >= nb) return r < 0;
    return path_cmp_exact(a, x, y, 0, &l) < 0;  // hashes differed, frames did not
  }
}

// Sort order: (gap, path) when a gap array is given (the new paths of a merge), else
// the path alone.
__device__ inline bool key_less(const CanonArgs &a, uint32_t x, uint32_t y) {
  if (x == kInf) return false;
  if (y == kInf) return true;
  if (a.gap) {
    const uint32_t gx = a.gap[x - a.id0], gy = a.gap[y - a.id0];
    if (gx != gy) return gx < gy;
  }
  return path_less(a, x, y);
}

// ---- sort -------------------------------------------------------------------------
// Block-local bitonic sort.  A merge's new paths carry their gap beside the key in LDS,
// so pairs in different gaps are ordered without a global load; only pairs in one gap
// compare paths.
__global__ __launch_bounds__(512) void sort_block_kernel(CanonArgs a, uint32_t *out) {
  __shared__ uint32_t key[kSortBlock];
  __shared__ uint32_t kgap[kSortBlock];
  const int tid = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * kSortBlock;
  for (int i = tid; i < kSortBlock; i += 512) {
    const bool in = base + i < a.d;
    key[i] = in ? (uint32_t)(a.id0 + base + i) : kInf;
    kgap[i] = in && a.gap ? a.gap[base + i] : 0u;
  }
  __syncthreads();
  for (int k = 2; k <= kSortBlock; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int i = 2 * j * (tid / j) + (tid % j), l = i + j;
      const uint32_t x = key[i], y = key[l], gx = kgap[i], gy = kgap[l];
      // ascending where (i & k) == 0: swap if y < x; else swap if x < y
      const bool up = (i & k) == 0;
      const uint32_t p = up ? y : x, q = up ? x : y, gp = up ? gy : gx, gq = up ? gx : gy;
      const bool swap = p != kInf && (q == kInf || (gp != gq ? gp < gq : path_less(a, p, q)));
      __syncthreads();
      if (swap) { key[i] = y; key[l] = x; kgap[i] = gy; kgap[l] = gx; }
      __syncthreads();
    }
  }
  for (int i = tid; i < kSortBlock; i += 512)
    if (base + i < a.d) out[base + i] = key[i];
}

__global__ __launch_bounds__(256) void merge_pass_kernel(CanonArgs a, const uint32_t *src, uint32_t *dst,
                                                         int64_t run) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t o0 = t * kMergeItems;
  if (o0 >= a.d) return;
  const int64_t pair = o0 / (2 * run), pb = pair * 2 * run;
  const int64_t la = min(run, a.d - pb), lb = max((int64_t)0, min(run, a.d - pb - run));
  const uint32_t *A = src + pb, *B = src + pb + la;
  const int64_t dgl = o0 - pb;
  int64_t lo = max((int64_t)0, dgl - lb), hi = min(dgl, la);
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (key_less(a, A[mid], B[dgl - 1 - mid])) lo = mid + 1; else hi = mid;
  }
  int64_t ia = lo, ib = dgl - lo;
  const int64_t cnt = min((int64_t)kMergeItems, la + lb - dgl);
  for (int64_t k = 0; k < cnt; ++k) {
    bool take_a;
    if (ia >= la) take_a = false;
    else if (ib >= lb) take_a = true;
    else take_a = !key_less(a, B[ib], A[ia]);
    dst[o0 + k] = take_a ? A[ia++] : B[ib++];
  }
}

// A merge's new paths: gap[j] = number of old paths (in their sorted order) below
// new path d_old + j.  Sixteen lanes search for one new path: each step compares it with
// 16 old paths that cut the remaining range into 17 parts (a 17-ary search), so the
// answer takes about log_17(d_old) rounds of path comparisons instead of log_2(d_old)
// (each comparison is a chain of dependent loads).
constexpr int kGapLanes = 16;
__global__ __launch_bounds__(256) void gap_kernel(CanonArgs a, const uint32_t *old_order, int64_t d_old, uint32_t *gap) {
  const int lane = threadIdx.x & 63, g = lane % kGapLanes, g0 = lane - g;
  const int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kGapLanes;
  const bool active = j < a.d - d_old;
  const uint32_t x = (uint32_t)(d_old + (active ? j : 0));
  // old_order[0, lo) are below x, old_order[hi, d_old) are not
  int64_t lo = 0, hi = active ? d_old : 0;
  for (;;) {
    const int64_t n = hi - lo;
    if (!__any(n > 0)) break;
    // pivot of this lane: every position when the range is at most 16 long, else the
    // 16 cuts into 17 parts (distinct and increasing for n >= 17)
    const int64_t pv = n <= kGapLanes ? lo + g : lo + (n * (g + 1)) / (kGapLanes + 1);
    const bool below = n > 0 && pv < hi && path_less(a, old_order[pv], x);
    const uint32_t m = (uint32_t)(__ballot(below) >> g0) & ((1u << kGapLanes) - 1);
    const int c = __popc(m);  // the pivots below x are a prefix (the old order is sorted)
    const int64_t p_lo = __shfl((long long)pv, g0 + (c > 0 ? c - 1 : 0), 64);
    const int64_t p_hi = __shfl((long long)pv, g0 + (c < kGapLanes ? c : kGapLanes - 1), 64);
    if (n > 0) {
      if (n <= kGapLanes) {
        lo += c;
        hi = lo;
      } else {
        const int64_t nlo = c > 0 ? p_lo + 1 : lo, nhi = c < kGapLanes ? p_hi : hi;
        lo = nlo;
        hi = nhi;
      }
    }
  }
  if (active && g == 0) gap[j] = (uint32_t)lo;
}

// Placement: the r-th new path (sorted by gap, then path) goes after its gap's old
// paths and the r new paths before it; old path i goes after the new paths whose
// gap is <= i.
__global__ __launch_bounds__(256) void place_new_kernel(const uint32_t *B, int64_t n_new, int64_t d_old,
                                                        const uint32_t *gap, uint32_t *gsorted, uint32_t *dst) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n_new) return;
  const uint32_t x = B[r];
  const uint32_t g = gap[x - d_old];
  gsorted[r] = g;
  dst[g + r] = x;
}
__global__ __launch_bounds__(256) void place_old_kernel(const uint32_t *A, int64_t d_old, const uint32_t *gsorted,
                                                        int64_t n_new, uint32_t *dst) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= d_old) return;
  int64_t lo = 0, hi = n_new;  // new paths with gap <= i
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if ((int64_t)gsorted[mid] <= i) lo = mid + 1; else hi = mid;
  }
  dst[i + lo] = A[i];
}

// ---- exact verification, lcp, scan rows ------------------------------------------------
__global__ void lcp_kernel(CanonArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i > a.d) return;
  const int C = 1 + a.m;
  if (i == a.d) { a.lcp[i] = 0; a.sparse[i] = 0; return; }
  // an order from a misleading hash may hold entries that are not path ids: they raise
  // the flag and read as path 0 here and in the kernels after this one
  uint32_t p = a.order[i];
  if (p >= (uint64_t)a.d) {
    atomicOr(&a.u_out[1], 1ull);
    p = 0;
    a.order[i] = 0;
  }
  uint32_t l = 0;
  if (i > 0) {
    uint32_t q = a.order[i - 1];
    if (q >= (uint64_t)a.d) q = 0;
    const int r = path_cmp_exact(a, q, p, 0, &l);
    if (r >= 0) atomicOr(&a.u_out[1], 1ull);  // not strictly increasing
  }
  a.lcp[i] = l;
  a.sparse[i] = l;  // level 0 of the range-minimum table
  uint64_t *row = a.scan_in + i * C;
  row[0] = (uint64_t)(a.plen[p] - l);
  for (int j = 0; j < a.m; ++j) row[1 + j] = a.psums[(int64_t)p * a.m + j];
}

// ---- multi-column exclusive scan (uint64, mod 2^64) -------------------------------------
__device__ inline uint64_t shfl_up_u64(uint64_t v, int o) {
  uint32_t lo = __shfl_up((uint32_t)v, o, 64), hi = __shfl_up((uint32_t)(v >> 32), o, 64);
  return ((uint64_t)hi << 32) | lo;
}

__global__ __launch_bounds__(256) void scan_reduce_kernel(const uint64_t *in, int64_t rows, int C, uint64_t *blk) {
  __shared__ uint64_t part[4];
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kScanRows;
  for (int c = 0; c < C; ++c) {
    uint64_t s = 0;
    for (int64_t r = r0 + tid; r < min(rows, r0 + kScanRows); r += 256) s += in[r * C + c];
    for (int o = 32; o > 0; o >>= 1) {
      uint32_t lo = __shfl_xor((uint32_t)s, o, 64), hi = __shfl_xor((uint32_t)(s >> 32), o, 64);
      s += ((uint64_t)hi << 32) | lo;
    }
    if ((tid & 63) == 0) part[tid >> 6] = s;
    __syncthreads();
    if (tid == 0) blk[blockIdx.x * C + c] = part[0] + part[1] + part[2] + part[3];
    __syncthreads();
  }
}

// exclusive scan of the block sums in place; totals into out row `rows`
__global__ __launch_bounds__(256) void scan_blocks_kernel(uint64_t *blk, int64_t nblk, int C, uint64_t *out,
                                                          int64_t rows) {
  __shared__ uint64_t part[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int c = 0; c < C; ++c) {
    uint64_t carry = 0;
    for (int64_t b0 = 0; b0 < nblk; b0 += 256) {
      const int64_t b = b0 + tid;
      const uint64_t v = b < nblk ? blk[b * C + c] : 0;
      uint64_t x = v;
      for (int o = 1; o < 64; o <<= 1) {
        const uint64_t y = shfl_up_u64(x, o);
        if (lane >= o) x += y;
      }
      if (lane == 63) part[wave] = x;
      __syncthreads();
      uint64_t before = carry;
      for (int w = 0; w < wave; ++w) before += part[w];
      if (b < nblk) blk[b * C + c] = before + x - v;
      const uint64_t tot = part[0] + part[1] + part[2] + part[3];
      __syncthreads();
      carry += tot;
    }
    if (tid == 0) out[rows * C + c] = carry;
  }
}

// direct: blk holds the raw block sums (not scanned), and each block adds up the sums of
// the blocks before it itself (at most kScanDirectBlocks of them); the last block also
// writes the totals row.  Otherwise blk holds their exclusive scan (scan_blocks_kernel).
constexpr int64_t kScanDirectBlocks = 4096;

__global__ __launch_bounds__(256) void scan_final_kernel(const uint64_t *in, int64_t rows, int C, const uint64_t *blk,
                                                         uint64_t *out, int direct) {
  __shared__ uint64_t part[4];
  __shared__ uint64_t pre;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kScanRows + tid * 4;
  for (int c = 0; c < C; ++c) {
    if (direct) {  // sum of the earlier blocks' sums of column c
      uint64_t x = 0;
      for (int64_t j = tid; j < (int64_t)blockIdx.x; j += 256) x += blk[j * C + c];
      for (int o = 32; o > 0; o >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)x, o, 64), hi = __shfl_xor((uint32_t)(x >> 32), o, 64);
        x += ((uint64_t)hi << 32) | lo;
      }
      if (lane == 0) part[wave] = x;
      __syncthreads();
      if (tid == 0) pre = part[0] + part[1] + part[2] + part[3];
      __syncthreads();
    }
    uint64_t v[4], s = 0;
    for (int k = 0; k < 4; ++k) {
      v[k] = r0 + k < rows ? in[(r0 + k) * C + c] : 0;
      s += v[k];
    }
    uint64_t x = s;
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t y = shfl_up_u64(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) part[wave] = x;
    __syncthreads();
    const uint64_t base = direct ? pre : blk[blockIdx.x * C + c];
    uint64_t run = base + x - s;
    for (int w = 0; w < wave; ++w) run += part[w];
    for (int k = 0; k < 4; ++k) {
      if (r0 + k < rows) out[(r0 + k) * C + c] = run;
      run += v[k];
    }
    if (direct && blockIdx.x == gridDim.x - 1 && tid == 0) out[rows * C + c] = base + part[0] + part[1] + part[2] + part[3];
    __syncthreads();
  }
}

// ---- range minima of lcp over [0, D] (lcp[D] = 0 is the sentinel) --------------------
__global__ void sparse_level_kernel(uint32_t *sp, int64_t n, int k) {
  // level k from level k-1 (k >= 1): minimum of lcp over [x, min(n, x + 2^k))
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= n) return;
  const uint32_t *prev = sp + (int64_t)(k - 1) * n;
  const int64_t h = (int64_t)1 << (k - 1);
  uint32_t v = prev[x];
  if (x + h < n) v = min(v, prev[x + h]);
  sp[(int64_t)k * n + x] = v;
}

// Levels top + 1 .. top + count in one launch: level k at x is the minimum of the
// level-top windows starting at x, x + 2^top, ... below x + 2^k (windows past n left
// out), so each thread reads 2^count - 1 level-top entries instead of waiting for the
// level below.
constexpr int kHighLevels = 7;  // levels per launch: 127 level-top reads per position
__global__ void sparse_high_kernel(uint32_t *sp, int64_t n, int top, int count) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= n) return;
  const uint32_t *lv = sp + (int64_t)top * n;
  const int64_t w = (int64_t)1 << top;
  uint32_t v = lv[x];
  for (int c = 1; c <= count; ++c) {
    // the new half of level top + c: windows x + 2^(top + c - 1) + j w, j < 2^(c - 1)
    const int64_t lo = x + (w << (c - 1));
    for (int64_t j = 0; j < ((int64_t)1 << (c - 1)); ++j) {
      const int64_t y = lo + j * w;
      if (y >= n) break;
      v = min(v, lv[y]);
    }
    sp[(int64_t)(top + c) * n + x] = v;
  }
}

// Levels 1 .. kTileLevels in one pass: a workgroup takes kTileOut positions, loads
// their lcp values and the 2^kTileLevels - 1 after them (past n: +inf) into LDS,
// and builds every level there from the one below.
constexpr int kTileLevels = 11, kTileOut = 2048, kTileIn = kTileOut + (1 << kTileLevels);
__global__ __launch_bounds__(1024) void sparse_tile_kernel(uint32_t *sp, const uint32_t *lcp, int64_t n, int top) {
  __shared__ uint32_t buf[2][kTileIn];
  const int64_t x0 = (int64_t)blockIdx.x * kTileOut;
  for (int i = threadIdx.x; i < kTileIn; i += 1024) buf[0][i] = x0 + i < n ? lcp[x0 + i] : 0xFFFFFFFFu;
  __syncthreads();
  int cur = 0;
  for (int k = 1; k <= top; ++k) {
    const int h = 1 << (k - 1);
    for (int i = threadIdx.x; i + h < kTileIn; i += 1024) buf[cur ^ 1][i] = min(buf[cur][i], buf[cur][i + h]);
    __syncthreads();
    cur ^= 1;
    for (int i = threadIdx.x; i < kTileOut; i += 1024)
      if (x0 + i < n) sp[(int64_t)k * n + x0 + i] = buf[cur][i];
  }
}

// first j >= s with lcp[j] < t (exists: lcp[D] = 0 < t for t >= 1).  Exponential search:
// skip blocks of 1, 2, 4, ... entries while a whole block is >= t, then descend within the
// block that holds the answer; about 2 log2(j - s) dependent loads instead of one per
// level, and most subtrees end a few paths on.
__device__ inline int64_t next_smaller(const CanonArgs &a, int64_t n, int64_t s, uint32_t t) {
  int64_t j = s;
  int k = 0;
  while (k < a.levels && j + ((int64_t)1 << k) <= n && a.sparse[(int64_t)k * n + j] >= t) {
    j += (int64_t)1 << k;
    ++k;
  }
  for (int q = k - 1; q >= 0; --q) {
    const int64_t w = (int64_t)1 << q;
    if (j + w <= n && a.sparse[(int64_t)q * n + j] >= t) j += w;
  }
  return j;
}
// largest j <= s with lcp[j] < t (exists: lcp[0] = 0 < t for t >= 1), the same search
// towards smaller indices
__device__ inline int64_t prev_smaller(const CanonArgs &a, int64_t n, int64_t s, uint32_t t) {
  int64_t j = s;
  int k = 0;
  while (k < a.levels && j - ((int64_t)1 << k) + 1 >= 0 && a.sparse[(int64_t)k * n + (j - ((int64_t)1 << k) + 1)] >= t) {
    j -= (int64_t)1 << k;
    ++k;
  }
  for (int q = k - 1; q >= 0; --q) {
    const int64_t w = (int64_t)1 << q;
    if (j - w + 1 >= 0 && a.sparse[(int64_t)q * n + (j - w + 1)] >= t) j -= w;
  }
  return j;
}

__device__ inline uint64_t node_base(const CanonArgs &a, int64_t i) { return 1 + a.scan_out[i * (1 + a.m)]; }

// chain parent of each path and the node -> path map.  The order is checked only after
// these kernels: if it is not a permutation (a misleading hash can repeat a path), the
// node count can exceed u_max, so nodes past it are not written and the order-violation
// flag is raised (the host then sorts again by exact comparisons).
__global__ void chain_kernel(CanonArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.d) return;
  const int64_t n = a.d + 1;
  const uint32_t L = a.lcp[i];
  uint32_t par = 0;
  if (L > 0) {
    const int64_t c = prev_smaller(a, n, i - 1, L);
    par = (uint32_t)(node_base(a, c) + L - a.lcp[c] - 1);
  }
  a.chain_parent[i] = par;
  const uint64_t b = node_base(a, i);
  const uint32_t cnt = a.plen[a.order[i]] - L;
  if (b + cnt > (uint64_t)a.u_max) {
    atomicOr(&a.u_out[1], 1ull);
    return;
  }
  if (cnt == 0) return;
  // the 64-node windows whose first node lies on this path (window 0 starts at node 1,
  // past the root)
  if (b == 1) a.win_path[0] = (uint32_t)i;
  for (uint64_t w = (b + 63) / 64; w <= (b + cnt - 1) / 64; ++w) a.win_path[w] = (uint32_t)i;
}

__global__ __launch_bounds__(256) void emit_kernel(CanonArgs a) {
  // a wave's 64 consecutive nodes stage their excl and incl rows in LDS ([2][256][m]
  // words), then write each array's 64 m words as one contiguous stretch
  extern __shared__ uint64_t emit_stage[];
  __shared__ uint32_t emit_mark[256];  // per wave: window position -> path offset
  const int C = 1 + a.m, m = a.m;
  const int lane = threadIdx.x & 63, w0 = threadIdx.x - lane;
  uint64_t *sx = emit_stage + (int64_t)w0 * m, *si = emit_stage + (int64_t)(256 + w0) * m;
  const int64_t n = a.d + 1;
  // (bounded by u_max, as in chain_kernel: past it the order is not a permutation)
  const int64_t U_all = (int64_t)(1 + a.scan_out[a.d * C]);
  const int64_t U = U_all < a.u_max ? U_all : a.u_max;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.u_out[0] = (unsigned long long)U;
    if (U_all > a.u_max) atomicOr(&a.u_out[1], 1ull);
  }
  uint32_t *mark = emit_mark + (w0 >> 6) * 64;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t base = (int64_t)blockIdx.x * blockDim.x + w0; base < U; base += stride) {
    const int64_t u = base + lane;
    // this window's paths: the one holding its first node and the 63 after it (every
    // path past the first has at least one node, so they cover the window); a node's
    // path is the last of them whose first node is at or before it
    // (window 0 holds only the root when there is no other node: no path to look up)
    int64_t i0 = (base > 0 || U > 1) ? (int64_t)a.win_path[base >> 6] : 0;
    if (i0 >= a.d && (base > 0 || U > 1)) {  // a window chain_kernel did not write (the order is not a permutation)
      if (lane == 0) atomicOr(&a.u_out[1], 1ull);
      i0 = 0;
    }
    const uint64_t nb = i0 + lane < a.d ? node_base(a, i0 + lane) : ~0ull;
    mark[lane] = 0;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    if (lane > 0 && nb >= (uint64_t)base && nb < (uint64_t)base + 64) mark[nb - base] = (uint32_t)lane;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    uint32_t off = mark[lane];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(off, o, 64);
      if (lane >= o) off = max(off, y);
    }
    const uint64_t bnode = ((uint64_t)__shfl((uint32_t)(nb >> 32), (int)off, 64) << 32) | __shfl((uint32_t)nb, (int)off, 64);
    if (u == 0) {
      a.parent[0] = kInf;
      a.frame[0] = 0;
      a.depth[0] = 0;
      a.subend[0] = (uint32_t)U;
      const bool empty_path = a.d > 0 && a.plen[a.order[0]] == 0;
      for (int j = 0; j < m; ++j) {
        sx[j] = empty_path ? a.psums[(int64_t)a.order[0] * m + j] : 0;
        si[j] = a.scan_out[a.d * C + 1 + j];
      }
    } else if (u < U) {
      int64_t i = i0 + (int64_t)off;
      uint64_t b = bnode;
      if (i >= a.d || b > (uint64_t)u) {  // (only when the order is not a permutation)
        atomicOr(&a.u_out[1], 1ull);
        i = 0;
        b = node_base(a, 0);
      }
      const uint32_t pid = a.order[i];
      const uint32_t L = a.lcp[i], len = a.plen[pid];
      uint32_t l = L + 1 + (uint32_t)(u - b);
      if (l > len || (uint64_t)u - b >= (uint64_t)len) {  // (only when the order is not a permutation)
        atomicOr(&a.u_out[1], 1ull);
        l = len;
      }
      a.parent[u] = u == (int64_t)b ? a.chain_parent[i] : (uint32_t)(u - 1);
      a.frame[u] = l ? a.pframes[a.pstart[pid] + l - 1] : 0u;
      a.depth[u] = l;
      const int64_t e = (i + 1 == a.d || l > a.lcp[i + 1]) ? i + 1 : next_smaller(a, n, i + 2, l);
      // the subtree is the paths i .. e-1 below depth l: ids up to the first node of path e
      a.subend[u] = (uint32_t)node_base(a, e);
      const uint64_t *pi = a.scan_out + i * C, *pe = a.scan_out + e * C;
      for (int j = 0; j < m; ++j) {
        sx[lane * m + j] = l == len ? a.psums[(int64_t)pid * m + j] : 0;
        si[lane * m + j] = pe[1 + j] - pi[1 + j];
      }
    }
    // every lane's LDS writes before any lane's reads
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    const int64_t words = (U - base < 64 ? U - base : 64) * m;
    for (int64_t k = lane; k < words; k += 64) {
      a.excl[base * m + k] = sx[k];
      a.incl[base * m + k] = si[k];
    }
    // every lane's reads before the next nodes' writes
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
  }
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_sort(CanonArgs &a, hipStream_t s) {
  if (a.d <= 0) return;
  uint32_t *src = a.order, *dst = a.order_tmp;
  hipLaunchKernelGGL(sort_block_kernel, dim3(blocks_for(a.d, kSortBlock)), dim3(512), 0, s, a, src);
  for (int64_t run = kSortBlock; run < a.d; run *= 2) {
    hipLaunchKernelGGL(merge_pass_kernel, dim3(blocks_for((a.d + kMergeItems - 1) / kMergeItems, 256)), dim3(256),
                       0, s, a, src, dst, run);
    uint32_t *t = src; src = dst; dst = t;
  }
  a.order = src;
  a.order_tmp = dst;
}

void launch_merge_order(CanonArgs &a, const uint32_t *old_order, int64_t d_old, uint32_t *scratch,
                        hipStream_t s) {
  const int64_t n_new = a.d - d_old;
  uint32_t *gap = scratch, *gsorted = scratch + n_new;
  const uint32_t *B = nullptr;
  uint32_t *dst = a.order;
  if (n_new > 0) {
    hipLaunchKernelGGL(gap_kernel, dim3(blocks_for(n_new * kGapLanes, 256)), dim3(256), 0, s, a, old_order, d_old, gap);
    CanonArgs r = a;
    r.d = n_new;
    r.id0 = d_old;
    r.gap = gap;
    launch_sort(r, s);  // new ids by (gap, path), in r.order (one of the two buffers)
    B = r.order;
    dst = r.order_tmp;
    hipLaunchKernelGGL(place_new_kernel, dim3(blocks_for(n_new, 256)), dim3(256), 0, s, B, n_new, d_old, gap,
                       gsorted, dst);
  }
  if (d_old > 0)
    hipLaunchKernelGGL(place_old_kernel, dim3(blocks_for(d_old, 256)), dim3(256), 0, s, old_order, d_old, gsorted,
                       n_new, dst);
  a.order_tmp = dst == a.order ? a.order_tmp : a.order;
  a.order = dst;
}

void launch_scan(const uint64_t *in, int64_t rows, int C, uint64_t *blk, uint64_t *out, hipStream_t s) {
  if (rows > 0) {
    const int64_t nblk = (rows + kScanRows - 1) / kScanRows;
    const int direct = nblk <= kScanDirectBlocks ? 1 : 0;
    hipLaunchKernelGGL(scan_reduce_kernel, dim3((unsigned)nblk), dim3(256), 0, s, in, rows, C, blk);
    if (!direct) hipLaunchKernelGGL(scan_blocks_kernel, dim3(1), dim3(256), 0, s, blk, nblk, C, out, rows);
    hipLaunchKernelGGL(scan_final_kernel, dim3((unsigned)nblk), dim3(256), 0, s, in, rows, C, blk, out, direct);
  } else {
    (void)hipMemsetAsync(out, 0, sizeof(uint64_t) * C, s);
  }
}

void launch_canon(const CanonArgs &a, hipStream_t s) {
  const int C = 1 + a.m;
  const int64_t n = a.d + 1;
  hipLaunchKernelGGL(lcp_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, a);
  launch_scan(a.scan_in, a.d, C, a.scan_blk, a.scan_out, s);
  // range-minimum table: level 0 (lcp itself) written by lcp_kernel, levels up to
  // kTileLevels in LDS tiles, the rest one level per launch
  const int top = std::min(a.levels - 1, kTileLevels);
  if (top >= 1)
    hipLaunchKernelGGL(sparse_tile_kernel, dim3(blocks_for(n, kTileOut)), dim3(1024), 0, s, a.sparse, a.lcp, n, top);
  if (top >= 1 && top < a.levels - 1) {
    const int count = std::min(a.levels - 1 - top, kHighLevels);
    hipLaunchKernelGGL(sparse_high_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, a.sparse, n, top, count);
    for (int k = top + count + 1; k < a.levels; ++k)
      hipLaunchKernelGGL(sparse_level_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, a.sparse, n, k);
  }
  if (a.d > 0) hipLaunchKernelGGL(chain_kernel, dim3(blocks_for(a.d, 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(emit_kernel, dim3(a.grid_nodes), dim3(256), (size_t)2 * 256 * a.m * 8, s, a);
}

}  // namespace cct
