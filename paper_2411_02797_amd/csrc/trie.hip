// Lexicographic order of the distinct full paths through a trie of 16-frame blocks.
//
// The canonical node ids are the lexicographic ranks of the paths (the paper's tree
// has no ids; see canon.hip).  Sorting variable-length paths by comparison needs long
// chains of dependent memory reads (paths share long prefixes), so the rank of each
// path is computed instead:
//   - every path of the path store is a chain of blocks of 16 frames (the last one
//     possibly shorter).  A block node is a distinct prefix ending at a block
//     boundary or at a path's end; nodes are deduplicated by hashing (the 16-frame
//     checkpoint hashes the store already holds) and then verified exactly: a node's
//     occurrences must share the parent node and the block's frames, which proves by
//     induction over the depth that equal nodes are equal prefixes;
//   - siblings (nodes with the same parent) are ordered by their blocks (frames
//     compared as unsigned, a shorter block first when it is a prefix of the other);
//   - with count(X) the number of paths through node X, the paths before path p are
//     those that leave p's chain X_1 .. X_n at an earlier sibling of some X_k, plus
//     the paths ending exactly at some X_{k-1} (proper prefixes of p):
//       rank(p) = sum_k [ sum of count(S) over siblings S < X_k  +  ends(X_{k-1}) ].
// A failed verification (a hash collision) or an oversized sibling group raises a
// flag, and the caller falls back to the comparison sort; the order is in any case
// re-verified frame by frame before it is used.
#include "common.h"

namespace cct {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kBlk = kStoreAlign;           // frames per block
constexpr int kChunk = 512;                 // groups up to this size are not split into buckets
constexpr int kSmallGroup = 64;             // groups up to this size are ranked by chunk
constexpr int kChunkCap = 2 * kChunk;       // staged members of one chunk (at most 2 kChunk - 1)
constexpr int kMedium = 2048;               // LDS sort capacity of one workgroup
constexpr uint64_t kRootSeed = 0x5851F42D4C957F2Dull;
constexpr uint16_t kNone = 0xFFFFu;
constexpr int kMaxBuckets = 256, kOversample = 2, kBucketTarget = 32;  // large groups (split_kernel)
// lists: buckets of up to 64 siblings (of large groups), groups of 65 .. 512 siblings,
// groups of more than 512, buckets of 65 .. 2048 siblings (of large groups)
enum { kListSmall = 0, kListMedium = 1, kListLarge = 2, kListMediumBucket = 3 };
constexpr int kFail = kTrieCtrFail;

__device__ inline void fail(const TrieArgs &a) { atomicOr(&a.ctr[kFail], 1ull); }

// Orders this wave's LDS accesses (every lane's earlier LDS writes before any lane's
// later LDS reads).
__device__ inline void wave_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

// block s of the store (frames [16 s, 16 s + 16)): its index k in its path, depth
// (prefix length at its end) and the path's length, from one word per block
struct BlockPos {
  uint32_t k, depth, len;
};
__device__ inline BlockPos block_pos(const TrieArgs &a, int64_t s) {
  const uint64_t w = a.bpos[s];
  BlockPos b;
  b.k = (uint32_t)w;
  b.len = (uint32_t)(w >> 32);
  b.depth = min((b.k + 1) * (uint32_t)kBlk, b.len);
  return b;
}
// frames in a node's block (1..16), from its depth
__device__ inline uint32_t block_frames(uint32_t depth) { return ((depth - 1) & (kBlk - 1)) + 1; }

// zero the node table, counts, end flags, child counts, bucket counts and counters
__global__ void clear_kernel(TrieArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= (int64_t)a.cap) {
    if (i < (int64_t)a.cap) { a.tkey[i] = 0; a.ncount[i] = 0; }
    a.nend[i] = 0;
    a.hist[i] = 0;
  }
  if (i < a.large_cap * kMaxBuckets) a.bcnt[i] = 0;
  if (i < 8) a.ctr[i] = 0;
}

__global__ void fill_kernel(TrieArgs a) {
  const int64_t d = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= a.d) return;
  a.order[d] = (uint32_t)d;
  const uint32_t len = a.plen[d];
  if (len == 0) {
    a.nend[a.cap] = 1;  // the empty path ends at the root
    return;
  }
  const int64_t b0 = a.pstart[d] / kBlk, nb = (len + kBlk - 1) / kBlk;
  for (int64_t k = 0; k < nb; ++k) a.bpos[b0 + k] = ((uint64_t)len << 32) | (uint64_t)k;
}

// Node of every block: open addressing on the prefix hash (claimed by CAS).
__global__ void insert_kernel(TrieArgs a) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.nblocks) return;
  const BlockPos b = block_pos(a, s);
  uint64_t key;
  if (b.depth == (b.k + 1) * kBlk) {
    key = a.pcp[s];  // full block: the checkpoint hash of the prefix
  } else {           // a path's last, partial block: hash it onto the previous checkpoint
    const uint32_t *f = a.pframes + s * kBlk;
    uint64_t acc = 0;
    for (uint32_t i = 0; i < b.depth - b.k * kBlk; ++i) acc += frame_term(f[i], b.k * kBlk + i);
    key = finish_hash(acc + (b.k ? a.pcp[s - 1] : kRootSeed) * 0x9E3779B97F4A7C15ull, b.depth);
  }
  if (key == 0) key = 1;
  const uint64_t mask = a.cap - 1;
  uint64_t slot = key & mask;
  for (uint64_t step = 0; step < a.cap; ++step) {
    uint64_t cur = a.tkey[slot];
    if (cur == 0) {
      cur = atomicCAS((unsigned long long *)&a.tkey[slot], 0ull, (unsigned long long)key);
      if (cur == 0) {
        a.tinfo[slot] = ((uint64_t)s << 32) | b.depth;
        a.occ[s] = (uint32_t)slot;
        return;
      }
    }
    if (cur == key) {
      a.occ[s] = (uint32_t)slot;
      return;
    }
    slot = (slot + 1) & mask;
  }
  a.occ[s] = 0;
  fail(a);
}

// Verify every occurrence against its node's representative (same depth, same parent
// node, same frames), link parents, count children per parent, paths per node (summed
// in an LDS map per workgroup first: nodes near the root are on many paths) and path
// ends.
constexpr int kLinkThreads = 1024, kLinkMap = 8192;
constexpr uint32_t kMapEmpty = 0xFFFFFFFFu;

__global__ __launch_bounds__(kLinkThreads) void link_kernel(TrieArgs a) {
  __shared__ uint32_t mkey[kLinkMap];
  __shared__ uint32_t mval[kLinkMap];
  __shared__ unsigned long long root_children;
  for (int i = threadIdx.x; i < kLinkMap; i += kLinkThreads) { mkey[i] = kMapEmpty; mval[i] = 0; }
  if (threadIdx.x == 0) root_children = 0;
  __syncthreads();
  const int64_t lo = (int64_t)blockIdx.x * a.nblocks / gridDim.x, hi = (int64_t)(blockIdx.x + 1) * a.nblocks / gridDim.x;
  for (int64_t s = lo + threadIdx.x; s < hi; s += kLinkThreads) {
    const BlockPos b = block_pos(a, s);
    const uint32_t X = a.occ[s];
    const uint64_t info = a.tinfo[X];
    const int64_t rep = (int64_t)(info >> 32);
    const uint32_t P = b.k ? a.occ[s - 1] : (uint32_t)a.cap;
    // the representative links the node and takes its index among its siblings (the
    // root's children, many, take theirs with one LDS atomic per wave)
    const bool is_rep = rep == s, to_root = P == (uint32_t)a.cap;
    const uint64_t rm = __ballot(is_rep && to_root);
    if (rm) {
      const int lane = threadIdx.x & 63, leader = __builtin_ctzll(rm);
      unsigned long long base = 0;
      if (lane == leader) base = atomicAdd(&root_children, (unsigned long long)__popcll(rm));
      base = __shfl(base, leader, 64);
      // (workgroup << 22) | index among this workgroup's root children
      if (is_rep && to_root) a.cidx[X] = (blockIdx.x << 22) | (uint32_t)(base + __popcll(rm & ((1ull << lane) - 1)));
    }
    if (is_rep) {
      a.nparent[X] = P;
      if (!to_root) a.cidx[X] = (uint32_t)atomicAdd((unsigned long long *)&a.hist[P], 1ull);
    } else {
      // a block's index in its path follows from its depth (16 k < depth <= 16 (k + 1)),
      // so the representative, of the same depth, has this block's index (and sits at
      // store block k or later: the guard keeps a slot no insertion wrote from reading
      // before the array)
      bool ok = (uint32_t)info == b.depth && rep < a.nblocks && rep >= (int64_t)b.k;
      if (ok) {
        const uint32_t RP = b.k ? a.occ[rep - 1] : (uint32_t)a.cap;
        ok = RP == P;
        if (ok) {
          const u32x4 *x = (const u32x4 *)(a.pframes + s * kBlk), *y = (const u32x4 *)(a.pframes + rep * kBlk);
          const uint32_t nf = b.depth - b.k * kBlk;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const u32x4 vx = x[c], vy = y[c];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if ((uint32_t)(4 * c + e) < nf && vx[e] != vy[e]) ok = false;
          }
        }
      }
      if (!ok) fail(a);
    }
    uint32_t h = hash32(X) & (kLinkMap - 1);
    bool done = false;
    for (int t = 0; t < 16 && !done; ++t) {
      uint32_t cur = mkey[h];
      if (cur == kMapEmpty) cur = atomicCAS(&mkey[h], kMapEmpty, X);
      if (cur == kMapEmpty || cur == X) {
        atomicAdd(&mval[h], 1u);
        done = true;
      } else {
        h = (h + 1) & (kLinkMap - 1);
      }
    }
    if (!done) atomicAdd(&a.ncount[X], 1u);
    if (b.depth == b.len) a.nend[X] = 1;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kLinkMap; i += kLinkThreads)
    if (mkey[i] != kMapEmpty) atomicAdd(&a.ncount[mkey[i]], mval[i]);
  // the root's children: this workgroup's block of indices (the root is one hot counter)
  if (threadIdx.x == 0)
    a.rootbase[blockIdx.x] = (uint32_t)(root_children ? atomicAdd((unsigned long long *)&a.hist[a.cap], root_children) : 0);
}

// Nodes grouped by parent: position = start of the parent's group (prefix sums of the
// child counts) + the node's index among its siblings.  Groups too large to be sorted
// by chunk are listed.
__global__ __launch_bounds__(256) void scatter_kernel(TrieArgs a) {
  const int64_t X = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (X >= (int64_t)a.cap || a.tkey[X] == 0) return;
  const uint32_t P = a.nparent[X], ci = a.cidx[X];
  const uint64_t c = P == (uint32_t)a.cap ? a.rootbase[ci >> 22] + (ci & ((1u << 22) - 1)) : ci;
  const uint64_t g0 = a.gstart[P], n = a.hist[P];
  const uint64_t pos = g0 + c;
  a.grouped[pos] = (uint32_t)X;
  a.posof[X] = (uint32_t)pos;
  if (c == 0 && n > (uint64_t)kChunk) {
    const unsigned long long i = atomicAdd(&a.ctr[kListLarge], 1ull);
    if ((int64_t)i < a.large_cap) {
      a.lists[kListLarge * a.list_cap + i] = (g0 << 32) | n;
      a.lgroup[P] = (uint32_t)i;
    } else {
      fail(a);
    }
  } else if (c == 0 && n > (uint64_t)kSmallGroup) {  // one workgroup each (medium_kernel)
    const unsigned long long i = atomicAdd(&a.ctr[kListMedium], 1ull);
    if ((int64_t)i < a.list_cap) a.lists[kListMedium * a.list_cap + i] = (g0 << 32) | n;
    else fail(a);
  }
}

// ---- sibling order ------------------------------------------------------------------
// a node's block: frames at the representative's store block, and their number
__device__ inline void node_block(const TrieArgs &a, uint32_t X, u32x4 (&v)[4], uint32_t &nf) {
  const uint64_t info = a.tinfo[X];
  const u32x4 *p = (const u32x4 *)(a.pframes + (info >> 32) * kBlk);
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = p[c];
  nf = block_frames((uint32_t)info);
}

// block x < block y: frames compared as unsigned over the shorter block, then the
// shorter block first.  Both rows are read whole (eight 16-byte LDS reads issued
// together); the first differing pair of frames is found without branches, and only its
// two frames are read again.  Frames past a block's end are zero in the store, and a
// difference there lies past the shorter block, which the length rule then decides.
__device__ inline bool block_less(const uint32_t *x, uint32_t nx, const uint32_t *y, uint32_t ny) {
  typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
  u64x2 a[4], b[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    a[c] = *(const u64x2 *)(x + 4 * c);
    b[c] = *(const u64x2 *)(y + 4 * c);
  }
  int fp = 8;  // first pair of frames that differs
#pragma unroll
  for (int p = 7; p >= 0; --p) fp = a[p >> 1][p & 1] != b[p >> 1][p & 1] ? p : fp;
  if (fp < 8) {
    const uint32_t i = 2 * fp + (x[2 * fp] == y[2 * fp] ? 1u : 0u);
    if (i < min(nx, ny)) return x[i] < y[i];
  }
  return nx < ny;
}

// A block's first two frames as one key.  Keys that differ order two blocks as
// block_less does: frame 0 decides if it differs; else frame 1 if both blocks have it;
// else one block has a single frame, its key's low word is the zero past its end, and
// the other block's frame 1 is then nonzero, so the key puts the shorter block first, as
// the length rule does.  Equal keys need the full comparison.  Keys live in an array of
// their own: a row's first word would put every key in one of two LDS banks.
__device__ inline uint64_t block_key(const u32x4 &v0) { return ((uint64_t)v0[0] << 32) | v0[1]; }

// the same order, for a block held in registers (y) against an LDS row (x)
__device__ inline bool block_less_seq(const uint32_t *x, uint32_t nx, const uint32_t *y, uint32_t ny) {
  const uint32_t n = min(nx, ny);
  for (uint32_t c = 0; c < 4 * 4; c += 4) {
    const u32x4 vx = *(const u32x4 *)(x + c), vy = *(const u32x4 *)(y + c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (c + e >= n) return nx < ny;
      if (vx[e] != vy[e]) return vx[e] < vy[e];
    }
  }
  return nx < ny;
}

// Bitonic sort of n <= 2 blockDim.x LDS entries: si holds entry indices, padded with
// kNone (+inf); lt(p, q) orders two entries.  Thread t takes pair t of every step; in
// a step of distance j <= 64 the pairs of wave w lie in entries [128 w, 128 w + 128),
// so between two such steps a wave waits only for its own LDS writes, and the
// workgroup meets at a barrier only around steps of longer distance.
template <class Less>
__device__ inline void lds_bitonic(uint16_t *si, int n, Less lt) {
  int n2 = 1;
  while (n2 < n) n2 <<= 1;
  for (int i = threadIdx.x; i < n2; i += blockDim.x) si[i] = i < n ? (uint16_t)i : kNone;
  __syncthreads();
  const int t = threadIdx.x;
  for (int k = 2; k <= n2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (t < n2 / 2) {
        const int i0 = 2 * j * (t / j) + (t % j), i1 = i0 + j;
        const uint16_t x = si[i0], y = si[i1];
        // ascending where (i0 & k) == 0, else descending: one comparison per pair, its
        // operands chosen by the direction (no divergence between the two)
        const bool asc = (i0 & k) == 0;
        const uint16_t p = asc ? y : x, q = asc ? x : y;
        if (p != kNone && (q == kNone || lt(p, q))) { si[i0] = y; si[i1] = x; }
      }
      const int j_next = j > 1 ? j >> 1 : k;  // the next step's distance (k: next stage)
      if (j <= 64 && j_next <= 64 && !(j == 1 && k == n2)) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_wave_barrier();
      } else {
        __syncthreads();
      }
    }
  }
}

constexpr int kMedThreads = 1024;
struct MedShared {
  uint32_t sb[kMedium][kBlk];
  uint64_t sk[kMedium];  // block keys (the splitter sample sort)
  uint8_t sn[kMedium];
  uint16_t si[kMedium];
};

// Groups of 2 .. 64 siblings, by chunk: workgroup c orders every such group whose
// start lies in positions [512 c, 512 c + 512) -- at most 575 consecutive positions,
// staged in LDS in position order, so every group is a contiguous run.  Each member's
// rank in its group is the number of siblings with a smaller block (siblings' blocks
// are distinct): at most 63 comparisons per member and no barriers between them.
struct ChunkShared {
  uint32_t sb[kChunkCap][kBlk];
  uint8_t sn[kChunkCap];
  uint16_t gs[kChunkCap];    // chunk-local start of the member's group (kNone: not ranked here)
  uint8_t gn[kChunkCap];     // the group's size
  uint32_t first, last_end;
};

constexpr int kChunkThreads = 512;
__global__ __launch_bounds__(kChunkThreads) void chunk_kernel(TrieArgs a) {
  __shared__ ChunkShared C;
  const uint64_t nodes = a.gstart[a.cap + 1];
  const uint64_t lo = (uint64_t)blockIdx.x * kChunk;
  if (lo >= nodes) return;
  if (threadIdx.x == 0) { C.first = 0xFFFFFFFFu; C.last_end = 0; }
  __syncthreads();
  {
    const uint64_t p = lo + threadIdx.x;
    if (threadIdx.x < kChunk && p < nodes) {
      const uint32_t P = a.nparent[a.grouped[p]];
      const uint64_t g0 = a.gstart[P], n = a.hist[P];
      if (g0 == p && n >= 2 && n <= (uint64_t)kSmallGroup) {
        atomicMin(&C.first, (uint32_t)p);
        atomicMax(&C.last_end, (uint32_t)(p + n));
      }
    }
  }
  __syncthreads();
  if (C.first == 0xFFFFFFFFu) return;
  const uint32_t first = C.first, m = C.last_end - first;
  // stage: position first + i with its group's local range (small groups only)
  constexpr int kPer = kChunkCap / kChunkThreads;
  uint32_t Xs[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const uint32_t i = threadIdx.x + q * kChunkThreads;
    Xs[q] = 0;
    if (i >= m) continue;
    const uint32_t X = a.grouped[first + i];
    const uint32_t P = a.nparent[X];
    const uint64_t g0 = a.gstart[P], n = a.hist[P];
    Xs[q] = X;
    C.gs[i] = kNone;
    if (n < 2 || n > (uint64_t)kSmallGroup || g0 < first || g0 + n > (uint64_t)first + m) continue;
    u32x4 v[4];
    uint32_t nf;
    node_block(a, X, v, nf);
#pragma unroll
    for (int c = 0; c < 4; ++c) *(u32x4 *)&C.sb[i][4 * c] = v[c];
    C.sn[i] = (uint8_t)nf;
    C.gs[i] = (uint16_t)(g0 - first);
    C.gn[i] = (uint8_t)n;
  }
  __syncthreads();
  // rank within the group; every original position was read before any write, and a
  // member's new position stays inside its group's range
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const uint32_t i = threadIdx.x + q * kChunkThreads;
    if (i >= m || C.gs[i] == kNone) continue;
    const uint32_t g = C.gs[i], n = C.gn[i];
    uint32_t rank = 0;
    for (uint32_t j = g; j < g + n; ++j)
      if (j != i && block_less(C.sb[j], C.sn[j], C.sb[i], C.sn[i])) ++rank;
    const uint32_t pos = first + g + rank;
    a.grouped[pos] = Xs[q];
    a.posof[Xs[q]] = pos;
  }
}

// Groups of 65 .. 512 siblings, or buckets of large groups of up to 2048 (list): one
// workgroup each, blocks in LDS.
__global__ __launch_bounds__(kMedThreads) void medium_kernel(TrieArgs a, int list) {
  __shared__ MedShared S;
  const uint64_t ng = min((uint64_t)a.ctr[list], (uint64_t)a.list_cap);
  // a bucket of a large group has its members in grouped2 (see rscatter_kernel)
  const uint32_t *src = list == kListMediumBucket ? a.grouped2 : a.grouped;
  for (uint64_t g = blockIdx.x; g < ng; g += gridDim.x) {
    const uint64_t e = a.lists[list * a.list_cap + g];
    const uint32_t start = (uint32_t)(e >> 32), n = (uint32_t)e;
    for (uint32_t i = threadIdx.x; i < n; i += kMedThreads) {
      u32x4 v[4];
      uint32_t nf;
      node_block(a, src[start + i], v, nf);
#pragma unroll
      for (int c = 0; c < 4; ++c) *(u32x4 *)&S.sb[i][4 * c] = v[c];
      S.sn[i] = (uint8_t)nf;
    }
    __syncthreads();
    lds_bitonic(S.si, (int)n, [&](uint16_t p, uint16_t q) { return block_less(S.sb[p], S.sn[p], S.sb[q], S.sn[q]); });
    // src[start + i] still holds the unsorted members (read before any write)
    uint32_t Xs[kMedium / kMedThreads];
    for (uint32_t i = threadIdx.x, q = 0; i < n; i += kMedThreads, ++q) Xs[q] = src[start + S.si[i]];
    __syncthreads();
    for (uint32_t i = threadIdx.x, q = 0; i < n; i += kMedThreads, ++q) {
      a.grouped[start + i] = Xs[q];
      a.posof[Xs[q]] = start + i;
    }
    __syncthreads();
  }
}

// Groups of more than 512 siblings are cut into ordered buckets: splitters from a
// sorted sample (2 per bucket, aiming at buckets of about 32), every member's bucket
// by binary search over the splitters, the group reordered by bucket; every bucket is
// then a group of its own, ordered by one wave (up to 64) or one workgroup.

__device__ inline int buckets_for(uint32_t n) {
  int nb = 2;
  while (nb < kMaxBuckets && (uint32_t)nb * kBucketTarget < n) nb <<= 1;
  return nb;
}

// one workgroup per large group: sorted sample -> splitters (node ids)
__global__ __launch_bounds__(kMedThreads) void split_kernel(TrieArgs a) {
  __shared__ MedShared S;
  const uint64_t ng = min((uint64_t)a.ctr[kListLarge], (uint64_t)a.large_cap);
  for (uint64_t g = blockIdx.x; g < ng; g += gridDim.x) {
    const uint64_t e = a.lists[kListLarge * a.list_cap + g];
    const uint32_t start = (uint32_t)(e >> 32), n = (uint32_t)e;
    const int nb = buckets_for(n), ns = nb * kOversample;
    for (int i = threadIdx.x; i < ns; i += kMedThreads) {
      const uint32_t X = a.grouped[start + (uint64_t)i * n / ns];
      u32x4 v[4];
      uint32_t nf;
      node_block(a, X, v, nf);
#pragma unroll
      for (int c = 0; c < 4; ++c) *(u32x4 *)&S.sb[i][4 * c] = v[c];
      S.sk[i] = block_key(v[0]);
      S.sn[i] = (uint8_t)nf;
    }
    __syncthreads();
    // a sample spread over a large group rarely shares its first two frames: keys first
    lds_bitonic(S.si, ns, [&](uint16_t p, uint16_t q) {
      const uint64_t kp = S.sk[p], kq = S.sk[q];
      return kp != kq ? kp < kq : block_less(S.sb[p], S.sn[p], S.sb[q], S.sn[q]);
    });
    // splitter j (j = 0 .. nb - 2) is the sample at sorted position (j + 1) * kOversample
    for (int j = threadIdx.x; j < nb - 1; j += kMedThreads)
      a.spl[g * kMaxBuckets + j] = a.grouped[start + (uint64_t)S.si[(j + 1) * kOversample] * n / ns];
    __syncthreads();
  }
}

// every member of a large group: its bucket (number of splitters below it), kept in
// posof until the member's position is known; bucket sizes counted per group
struct ClassShared {
  uint32_t sb[2][kMaxBuckets][kBlk];
  uint8_t sn[2][kMaxBuckets];
  uint32_t grp[2];
};
__global__ __launch_bounds__(kMedThreads) void classify_kernel(TrieArgs a) {
  __shared__ ClassShared C;
  const uint64_t nodes = a.gstart[a.cap + 1];
  const uint64_t lo = (uint64_t)blockIdx.x * kChunk;
  if (lo >= nodes) return;
  const uint64_t p = lo + threadIdx.x;
  uint32_t X = 0, P = 0, g = 0xFFFFFFFFu;
  if (threadIdx.x < kChunk && p < nodes) {
    X = a.grouped[p];
    P = a.nparent[X];
    if (a.hist[P] > (uint64_t)kChunk) {
      g = a.lgroup[P];  // listed large group (an unlisted one has already failed the call)
      if ((uint64_t)g >= min((uint64_t)a.ctr[kListLarge], (uint64_t)a.large_cap)) g = 0xFFFFFFFFu;
    }
  }
  // at most two large groups overlap 1024 consecutive positions: the first and last
  // position's
  if (threadIdx.x == 0) { C.grp[0] = 0xFFFFFFFFu; C.grp[1] = 0xFFFFFFFFu; }
  __syncthreads();
  const uint64_t last = min(lo + kChunk, nodes) - 1;
  if (p == lo) C.grp[0] = g;
  if (p == last) C.grp[1] = g;
  __syncthreads();
  for (int h = 0; h < 2; ++h) {
    const uint32_t gh = C.grp[h];
    if (gh == 0xFFFFFFFFu) continue;
    const uint64_t e = a.lists[kListLarge * a.list_cap + gh];
    const int nb = buckets_for((uint32_t)e);
    for (int j = threadIdx.x; j < nb - 1; j += kMedThreads) {
      u32x4 v[4];
      uint32_t nf;
      node_block(a, a.spl[gh * kMaxBuckets + j], v, nf);
#pragma unroll
      for (int c = 0; c < 4; ++c) *(u32x4 *)&C.sb[h][j][4 * c] = v[c];
      C.sn[h][j] = (uint8_t)nf;
    }
  }
  __syncthreads();
  if (g == 0xFFFFFFFFu) return;
  const int h = g == C.grp[0] ? 0 : 1;
  const int nb = buckets_for((uint32_t)a.lists[kListLarge * a.list_cap + g]);
  u32x4 v[4];
  uint32_t nf;
  node_block(a, X, v, nf);
  uint32_t x[kBlk];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int q = 0; q < 4; ++q) x[4 * c + q] = v[c][q];
  int blo = 0, bhi = nb - 1;
  while (blo < bhi) {
    const int mid = (blo + bhi) >> 1;
    if (block_less_seq(C.sb[h][mid], C.sn[h][mid], x, nf)) blo = mid + 1; else bhi = mid;
  }
  a.posof[X] = (uint32_t)blo;
  atomicAdd(&a.bcnt[g * kMaxBuckets + blo], 1u);
}

// Large groups reordered by bucket, in two grid-wide steps (a large group has
// thousands of members):
//  - bstart_kernel, one small workgroup per large group: bucket starts (exclusive
//    prefix sums of the bucket sizes, into spl, whose splitters are no longer needed),
//    every non-empty bucket listed for sorting, and the sizes reset to serve as cursors;
//  - rscatter_kernel, every member: its bucket's start + a cursor atomic, into grouped2.
// The kernels that order the buckets read their members from grouped2 and write the
// final positions into grouped (a member still being read from grouped by rscatter
// cannot be overwritten there).
__global__ __launch_bounds__(kMaxBuckets) void bstart_kernel(TrieArgs a) {
  __shared__ uint32_t wsum[kMaxBuckets / 64];
  __shared__ uint32_t wlist[2][kMaxBuckets / 64];  // per wave: its buckets' offset in each list
  __shared__ unsigned long long lbase[2];
  const uint64_t ng = min((uint64_t)a.ctr[kListLarge], (uint64_t)a.large_cap);
  const uint64_t g = blockIdx.x;
  if (g >= ng) return;
  const uint64_t e = a.lists[kListLarge * a.list_cap + g];
  const uint32_t start = (uint32_t)(e >> 32), n = (uint32_t)e;
  const int nb = buckets_for(n);
  const int j = threadIdx.x, lane = j & 63, w = j >> 6;
  const uint32_t c = j < nb ? a.bcnt[g * kMaxBuckets + j] : 0u;
  uint32_t x = c;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  // every non-empty bucket is listed (a bucket of one too: its member's position is
  // written by bucket_kernel), the small ones and the medium ones in lists of their own;
  // the workgroup reserves its entries in each list with one atomic (every large group
  // appends up to 256 buckets at the same time)
  const bool small = j < nb && c >= 1 && c <= 64, medium = j < nb && c > 64 && c <= (uint32_t)kMedium;
  const uint64_t ms = __ballot(small), mm = __ballot(medium);
  if (lane == 0) { wlist[0][w] = (uint32_t)__popcll(ms); wlist[1][w] = (uint32_t)__popcll(mm); }
  __syncthreads();
  if (j == 0) {
    uint32_t ts = 0, tm = 0;
    for (int q = 0; q < kMaxBuckets / 64; ++q) {
      const uint32_t cs = wlist[0][q], cm = wlist[1][q];
      wlist[0][q] = ts; wlist[1][q] = tm;
      ts += cs; tm += cm;
    }
    lbase[0] = ts ? atomicAdd(&a.ctr[kListSmall], (unsigned long long)ts) : 0;
    lbase[1] = tm ? atomicAdd(&a.ctr[kListMediumBucket], (unsigned long long)tm) : 0;
  }
  __syncthreads();
  uint32_t before = 0;
  for (int q = 0; q < w; ++q) before += wsum[q];
  const uint32_t bs = before + x - c;
  if (j >= nb) return;
  a.spl[g * kMaxBuckets + j] = bs;
  a.bcnt[g * kMaxBuckets + j] = 0;
  if (c > (uint32_t)kMedium) { fail(a); return; }
  if (!small && !medium) return;
  const int cls = small ? 0 : 1;
  const uint64_t below = (small ? ms : mm) & ((1ull << lane) - 1);
  const unsigned long long i = lbase[cls] + wlist[cls][w] + (unsigned long long)__popcll(below);
  const int list = small ? kListSmall : kListMediumBucket;
  if ((int64_t)i < a.list_cap) a.lists[list * a.list_cap + i] = ((uint64_t)(start + bs) << 32) | c;
  else fail(a);
}

// the large group of the member at position p (its bucket is in posof), or -1
__device__ inline int64_t large_group_of(const TrieArgs &a, uint32_t X) {
  const uint32_t P = a.nparent[X];
  if (a.hist[P] <= (uint64_t)kChunk) return -1;
  const uint64_t g = a.lgroup[P];
  return g < min((uint64_t)a.ctr[kListLarge], (uint64_t)a.large_cap) ? (int64_t)g : -1;
}

__global__ void rscatter_kernel(TrieArgs a) {
  const uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= a.gstart[a.cap + 1]) return;
  const uint32_t X = a.grouped[p];
  const int64_t g = large_group_of(a, X);
  if (g < 0) return;
  const uint32_t bk = a.posof[X];
  const uint64_t dst = a.gstart[a.nparent[X]] + a.spl[g * kMaxBuckets + bk] + atomicAdd(&a.bcnt[g * kMaxBuckets + bk], 1u);
  a.grouped2[dst] = X;
}

// buckets of 1 .. 64 of large groups (members in grouped2): one wave each, every member
// counts the members before it
constexpr int kBucketWaves = 4;
__global__ __launch_bounds__(64 * kBucketWaves) void bucket_kernel(TrieArgs a) {
  __shared__ uint32_t sb[kBucketWaves][64][kBlk];
  __shared__ uint32_t sn[kBucketWaves][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t ng = min((uint64_t)a.ctr[kListSmall], (uint64_t)a.list_cap);
  for (uint64_t g = (uint64_t)blockIdx.x * kBucketWaves + w; g < ng; g += (uint64_t)gridDim.x * kBucketWaves) {
    const uint64_t e = a.lists[kListSmall * a.list_cap + g];
    const uint32_t start = (uint32_t)(e >> 32), n = (uint32_t)e;
    uint32_t X = 0;
    if (lane < (int)n) {
      X = a.grouped2[start + lane];
      u32x4 v[4];
      uint32_t nf;
      node_block(a, X, v, nf);
#pragma unroll
      for (int c = 0; c < 4; ++c) *(u32x4 *)&sb[w][lane][4 * c] = v[c];
      sn[w][lane] = nf;
    }
    wave_sync();
    if (lane < (int)n) {
      uint32_t rank = 0;
      for (uint32_t j = 0; j < n; ++j)
        if (j != (uint32_t)lane && block_less(sb[w][j], sn[w][j], sb[w][lane], sn[w][lane])) ++rank;
      a.grouped[start + rank] = X;
      a.posof[X] = start + rank;
    }
    wave_sync();
  }
}

// path counts in grouped order (zero past the last node)
__global__ void counts_kernel(TrieArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.nblocks) return;
  const uint64_t nodes = a.gstart[a.cap + 1];
  a.cnt[i] = (uint64_t)i < nodes ? a.ncount[a.grouped[i]] : 0;
}

// Eight lanes per path: lane g takes the path's blocks g, g + 8, ...; a block's term
// needs only its own node and the node before it, so the terms of one path load in
// parallel and meet by three shuffles within the eight lanes.
constexpr int kRankLanes = 8;
__global__ __launch_bounds__(256) void rank_kernel(TrieArgs a) {
  const int64_t d = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kRankLanes;
  const int g = threadIdx.x % kRankLanes;
  const bool active = d < a.d;
  const uint32_t len = active ? a.plen[d] : 0u;
  const int64_t b0 = active ? a.pstart[d] / kBlk : 0, nb = (len + kBlk - 1) / kBlk;
  uint64_t part = 0;
  for (int64_t k = g; k < nb; k += kRankLanes) {
    const uint32_t X = a.occ[b0 + k];
    const uint32_t prev = k ? a.occ[b0 + k - 1] : (uint32_t)a.cap;
    part += a.cnt_scan[a.posof[X]] - a.cnt_scan[a.gstart[a.nparent[X]]] + a.nend[prev];
  }
#pragma unroll
  for (int o = kRankLanes / 2; o > 0; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)part, o, 64), hi = __shfl_xor((uint32_t)(part >> 32), o, 64);
    part += ((uint64_t)hi << 32) | lo;
  }
  if (!active || g != 0) return;
  if (part < (uint64_t)a.d) a.order[part] = (uint32_t)d;
  else fail(a);
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

void launch_trie_sort(const TrieArgs &a, hipStream_t s, hipStream_t s2, hipEvent_t fork, hipEvent_t mid,
                      hipEvent_t join) {
  if (a.d <= 0) return;
  const bool two = s2 != s && fork && join;
  hipLaunchKernelGGL(clear_kernel, dim3(blocks_for((int64_t)a.cap + 1, 256)), dim3(256), 0, s, a);
  hipLaunchKernelGGL(fill_kernel, dim3(blocks_for(a.d, 256)), dim3(256), 0, s, a);
  if (a.nblocks > 0) {
    hipLaunchKernelGGL(insert_kernel, dim3(blocks_for(a.nblocks, 256)), dim3(256), 0, s, a);
    const int64_t link_grid = std::max<int64_t>(1, std::min<int64_t>(blocks_for(a.nblocks, 1024), 512));
    hipLaunchKernelGGL(link_kernel, dim3((unsigned)link_grid), dim3(kLinkThreads), 0, s, a);
    launch_scan(a.hist, (int64_t)a.cap + 1, 1, a.scan_blk, a.gstart, s);
    hipLaunchKernelGGL(scatter_kernel, dim3(blocks_for((int64_t)a.cap, 256)), dim3(256), 0, s, a);
    // Sibling order.  Small groups (chunk_kernel) and the listed groups of 65 .. 512
    // (medium_kernel) touch only their own positions; the large groups' pipeline (split,
    // classify, bucket scatter, then its buckets) reads the other positions only to see
    // that they are not in a large group, which any member of the same group tells.  So
    // the two run side by side, on two streams when the caller gives a second one.
    hipStream_t sa = s;
    if (two && hipEventRecord(fork, s) == hipSuccess && hipStreamWaitEvent(s2, fork, 0) == hipSuccess) sa = s2;
    hipLaunchKernelGGL(chunk_kernel, dim3(blocks_for(a.nblocks, kChunk)), dim3(kChunkThreads), 0, sa, a);
    hipLaunchKernelGGL(medium_kernel, dim3(256), dim3(kMedThreads), 0, sa, a, (int)kListMedium);
    hipLaunchKernelGGL(split_kernel, dim3(256), dim3(kMedThreads), 0, s, a);
    hipLaunchKernelGGL(classify_kernel, dim3(blocks_for(a.nblocks, kChunk)), dim3(kMedThreads), 0, s, a);
    hipLaunchKernelGGL(bstart_kernel, dim3((unsigned)a.large_cap), dim3(kMaxBuckets), 0, s, a);
    hipLaunchKernelGGL(rscatter_kernel, dim3(blocks_for(a.nblocks, 256)), dim3(256), 0, s, a);
    // the buckets of up to 64 and the larger ones are disjoint: the small ones follow the
    // side branch once the scatter is done
    hipStream_t sb = s;
    if (sa != s && mid && hipEventRecord(mid, s) == hipSuccess && hipStreamWaitEvent(sa, mid, 0) == hipSuccess) sb = sa;
    hipLaunchKernelGGL(bucket_kernel, dim3(1024), dim3(64 * kBucketWaves), 0, sb, a);
    hipLaunchKernelGGL(medium_kernel, dim3(256), dim3(kMedThreads), 0, s, a, (int)kListMediumBucket);
    if (sa != s && (hipEventRecord(join, sa) != hipSuccess || hipStreamWaitEvent(s, join, 0) != hipSuccess)) {
      // the side branch cannot be joined: wait for it from the host before going on
      (void)hipGetLastError();
      (void)hipStreamSynchronize(sa);
    }
    hipLaunchKernelGGL(counts_kernel, dim3(blocks_for(a.nblocks, 256)), dim3(256), 0, s, a);
    launch_scan(a.cnt, a.nblocks, 1, a.scan_blk, a.cnt_scan, s);
  }
  hipLaunchKernelGGL(rank_kernel, dim3(blocks_for(a.d * kRankLanes, 256)), dim3(256), 0, s, a);
}

}  // namespace cct
