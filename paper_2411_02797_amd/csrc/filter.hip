// Analysis queries as data-parallel filters over the tree.  The paper's example analyses
// walk the tree and flag nodes whose metric ratio crosses a threshold: a kernel whose
// time is a large share of the root's (hotspot), a frame whose GPU time per kernel is
// small (kernel fusion), a frame whose CPU time is large against its GPU time (CPU
// latency) (Implementation, "Performance Analyzer", "Example Analyses").
//
// One predicate covers them: node v matches when a(v) / b(v) is above (or below) the
// threshold p / q, tested without division as a(v) * q > p * b(v) (or <) in exact 128-bit
// integer arithmetic; a(v) is one of the node's sums, b(v) is 1, another of the node's
// sums, or the root's inclusive sum.  Optionally only leaves (nodes without children)
// match.
//
// Two passes over tiles of kFilterTile nodes list the matches in ascending id order
// (preorder): the first evaluates the predicate once per node and keeps it as one bit
// (a wave's ballot is the mask word of its 64 nodes) plus a match count per tile; one
// workgroup scans the tile counts (a few thousand for millions of nodes); the second pass
// reads only the mask and writes each match's id at its tile's offset plus its rank among
// the tile's earlier matches.
#include <mutex>

#include "common.h"

namespace cct {

namespace {

constexpr int kFilterThreads = 256;
constexpr int kFilterRounds = kFilterTile / kFilterThreads;  // nodes per thread in the first pass
constexpr int kTileWords = kFilterTile / 64;                 // mask words per tile
constexpr int kScanThreads = 1024, kScanPer = 4;             // tile-count scan: one workgroup
static_assert(kFilterTile % kFilterThreads == 0 && kTileWords <= 64, "tile shape");

// a * q versus p * b over unsigned 128-bit products: -1, 0, +1
__device__ inline int cmp_products(uint64_t a, uint64_t q, uint64_t p, uint64_t b) {
  const uint64_t lo1 = a * q, hi1 = __umul64hi(a, q);
  const uint64_t lo2 = p * b, hi2 = __umul64hi(p, b);
  if (hi1 != hi2) return hi1 < hi2 ? -1 : 1;
  if (lo1 != lo2) return lo1 < lo2 ? -1 : 1;
  return 0;
}

__device__ inline bool node_matches(const FilterArgs &a, int64_t v) {
  const uint64_t *num = a.num_excl ? a.excl : a.incl;
  const uint64_t x = num[v * a.m + a.num_metric];
  uint64_t y = 1;
  if (a.den_kind == kDenMetric) y = (a.den_excl ? a.excl : a.incl)[v * a.m + a.den_metric];
  else if (a.den_kind == kDenRoot) y = a.incl[a.den_metric];
  const int c = cmp_products(x, a.thr_den, a.thr_num, y);
  const bool hit = a.op > 0 ? c > 0 : c < 0;
  return hit && (!a.leaves_only || a.subend[v] == (uint32_t)(v + 1));  // a leaf's subtree is itself
}

// mask[w] bit l: node 64 w + l matches (every word of every tile is written, zero past U);
// count[t]: matches in tile t
__global__ __launch_bounds__(kFilterThreads) void filter_mask_kernel(FilterArgs a, uint64_t *mask, uint32_t *count) {
  __shared__ uint32_t wave_count[kFilterThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kFilterTile;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  bool hit[kFilterRounds];
#pragma unroll
  for (int r = 0; r < kFilterRounds; ++r) {
    const int64_t v = base + r * kFilterThreads + threadIdx.x;
    hit[r] = v < a.u && node_matches(a, v);
  }
  uint32_t c = 0;
#pragma unroll
  for (int r = 0; r < kFilterRounds; ++r) {
    const uint64_t bits = __ballot(hit[r]);
    c += (uint32_t)__popcll(bits);
    if (lane == 0) mask[(base + r * kFilterThreads + wave * 64) >> 6] = bits;
  }
  if (lane == 0) wave_count[wave] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kFilterThreads / 64; ++w) t += wave_count[w];
    count[blockIdx.x] = t;
  }
}

// pos[t] = count[0] + ... + count[t - 1] for t <= T (pos[T]: all matches); a single
// workgroup walks the counts kScanThreads * kScanPer at a time
__global__ __launch_bounds__(kScanThreads) void filter_scan_kernel(const uint32_t *count, int64_t T, uint64_t *pos) {
  __shared__ uint32_t wave_sum[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t carry = 0;
  for (int64_t t0 = 0; t0 < T; t0 += kScanThreads * kScanPer) {
    const int64_t t = t0 + (int64_t)tid * kScanPer;
    uint32_t c[kScanPer], mine = 0;
#pragma unroll
    for (int k = 0; k < kScanPer; ++k) {
      c[k] = t + k < T ? count[t + k] : 0;
      mine += c[k];
    }
    uint32_t x = mine;  // inclusive scan over the wave
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane == 63) wave_sum[wave] = x;
    __syncthreads();
    uint32_t before = 0, total = 0;  // at most kFilterTile * kScanThreads * kScanPer < 2^32
    for (int w = 0; w < kScanThreads / 64; ++w) {
      const uint32_t v = wave_sum[w];
      before += w < wave ? v : 0;
      total += v;
    }
    uint64_t run = carry + before + (x - mine);
#pragma unroll
    for (int k = 0; k < kScanPer; ++k) {
      if (t + k < T) pos[t + k] = run;
      run += c[k];
    }
    carry += total;
    __syncthreads();  // wave_sum is rewritten by the next round
  }
  if (tid == 0) pos[T] = carry;
}

// one wave per tile: lanes below kTileWords hold the tile's mask words and an inclusive
// scan of their bit counts; then word by word, each set bit's lane writes its node id
__global__ __launch_bounds__(64) void filter_write_kernel(const uint64_t *mask, const uint64_t *pos, int64_t capacity,
                                                          int64_t *out) {
  const int64_t tile = blockIdx.x;
  const int lane = threadIdx.x;
  const uint64_t mine = lane < kTileWords ? mask[tile * kTileWords + lane] : 0;
  int incl = __popcll(mine);
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(incl, d);
    if (lane >= d) incl += t;
  }
  const int64_t base = (int64_t)pos[tile];
  if (base >= capacity) return;  // uniform across the wave
  const uint64_t below = (1ull << lane) - 1;
  for (int j = 0; j < kTileWords; ++j) {
    const uint32_t lo = __shfl((uint32_t)mine, j), hi = __shfl((uint32_t)(mine >> 32), j);
    const uint64_t word = ((uint64_t)hi << 32) | lo;
    const int before = __shfl(incl, j) - __popcll(word);  // matches of the tile's earlier words
    if ((word >> lane) & 1) {
      const int64_t k = base + before + __popcll(word & below);
      if (k < capacity) out[k] = tile * kFilterTile + j * 64 + lane;
    }
  }
}

// Scratch of the filter entry point that allocates nothing: the mask words, tile counts
// and tile offsets of up to kFilterStaticTiles tiles, laid out as filter_static_layout
// says.  Each GPU holds its own copy for the life of the process; every call on a GPU
// reuses it, so calls that overlap on one GPU race.  Host code never uses this name as an
// address (on the host it only stands for the symbol): the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[kFilterStaticBytes];

}  // namespace

int64_t filter_tiles(int64_t u) { return (u + kFilterTile - 1) / kFilterTile; }

FilterScratch filter_static_layout(void *base) {
  unsigned char *b = static_cast<unsigned char *>(base);
  FilterScratch f;
  f.mask = reinterpret_cast<uint64_t *>(b);
  f.count = reinterpret_cast<uint32_t *>(b + kFilterStaticTiles * kTileWords * 8);
  f.pos = reinterpret_cast<uint64_t *>(b + kFilterStaticTiles * (kTileWords * 8 + 4));
  return f;
}
static_assert(kFilterStaticTiles * (kTileWords * 8 + 4 + 8) + 8 <= kFilterStaticBytes, "static filter scratch");
static_assert((kFilterStaticTiles * (kTileWords * 8 + 4)) % 8 == 0, "pos alignment");

void *filter_static_scratch() {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *ptr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    ptr[dev] = p;
  }
  return ptr[dev];
}

void launch_filter_mask(const FilterArgs &a, uint64_t *mask, uint32_t *count, hipStream_t s) {
  const int64_t tiles = filter_tiles(a.u);
  if (tiles > 0)
    hipLaunchKernelGGL(filter_mask_kernel, dim3((unsigned)tiles), dim3(kFilterThreads), 0, s, a, mask, count);
}

void launch_filter_scan(const uint32_t *count, int64_t tiles, uint64_t *pos, hipStream_t s) {
  hipLaunchKernelGGL(filter_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, count, tiles, pos);
}

void launch_filter_write(int64_t u, const uint64_t *mask, const uint64_t *pos, int64_t capacity, int64_t *out,
                         hipStream_t s) {
  const int64_t tiles = filter_tiles(u);
  if (tiles > 0 && capacity > 0)
    hipLaunchKernelGGL(filter_write_kernel, dim3((unsigned)tiles), dim3(64), 0, s, mask, pos, capacity, out);
}

}  // namespace cct
