// Internal definitions shared by the HIP kernels and the host runtime of libcct.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cct {

// ---- unique-path table -------------------------------------------------------
// One 16-byte entry per slot.  word = (tag << 32) | ref, where ref is a path id of the
// tree's path store, or kEventRef | event index for a path first seen in the current
// call; it is claimed with one 64-bit CAS.  info tells where the slot's frames live and
// how many there are, so a lookup needs one memory round trip: written by the claimer
// right after its CAS (readers that still see kEmptyInfo fall back to ref).
struct Slot {
  uint64_t word;
  uint64_t info;
};
constexpr uint64_t kEmptySlot = ~0ull;
constexpr uint64_t kEmptyInfo = ~0ull;
constexpr uint32_t kEventRef = 0x80000000u;
constexpr uint32_t kRefMask = 0x7FFFFFFFu;
// info = (first frame << 24) | (in path store << 23) | length; lengths >= kInfoLongLen
// are stored as kInfoLongLen (their exact length is then read through ref).
constexpr uint64_t kInfoLongLen = 0x7FFFFF;
__host__ __device__ inline uint64_t make_info(uint64_t base, bool store, uint64_t len) {
  return (base << 24) | ((uint64_t)store << 23) | (len < kInfoLongLen ? len : kInfoLongLen);
}

// ---- ingest tiling -------------------------------------------------------------
constexpr int kIngestThreads = 1024;    // 16 waves of 64 (4 per SIMD), each with its own tile loop
constexpr int kWaveEvents = 63;         // max events per wave tile (lane j holds offset j, j <= 63)
constexpr int kLaneBlocks = 2;          // 16-frame blocks held by each lane of a wave tile
constexpr int kWaveFrames = 64 * 16 * kLaneBlocks;  // frames of a wave tile
constexpr int kCacheEntries = 4096;     // LDS resolved-path cache entries per workgroup

// ---- counters written by the ingest kernels --------------------------------------
enum Counter { kCtrNew = 0, kCtrNewFrames = 1, kCtrError = 2, kCtrOverflow = 3, kCtrNewLen = 4,
               kCtrCount = 8 };
enum ErrorBits { kErrOffsets = 1 };
constexpr uint32_t kNoSlot = 0xFFFFFFFFu;  // event not resolved (the call fails or retries)

// ---- path hashing ----------------------------------------------------------------
// Checkpoint hashes (prefixes at 16-frame boundaries, used to order paths) are a sum
// over the frames of a term of (frame, position), so partial sums over any split of
// the path combine by addition; a murmur3-style finalizer mixes in the length.  The
// term is one 32 x 32 -> 64-bit product of two position-dependent mixes of the frame;
// both factors move with the position, so paths over a few small frame ids still
// spread.  Correctness never depends on a hash: every match is verified frame by frame.
constexpr uint32_t kTermMulX = 0x9E3779B9u, kTermMulY = 0x85EBCA6Bu, kTermXorY = 0x5BD1E995u;
__host__ __device__ inline uint64_t frame_term(uint32_t f, uint32_t k) {
  const uint32_t x = f + k * kTermMulX;
  const uint32_t y = (f ^ kTermXorY) + k * kTermMulY;
  return (uint64_t)x * (uint64_t)(y | 1u);
}
// The unique-path table hashes pairs of frames instead.  A path of len frames is cut
// into ceil(len / 16) blocks of 16 frames: block m starts at frame 16 m, except that
// the last block of a path of 16 frames or more ends at the path's end (so it overlaps
// the block before it when len is not a multiple of 16; a path shorter than 16 frames
// is one block, zero-padded).  Pair i of block m, (F[s + 2i], F[s + 2i + 1]) with s the
// block's first frame, is pair p = 8 m + i and contributes
//   (F[s + 2i] + p*kPairMulX + kPairAddX) * (F[s + 2i + 1] + p*kPairMulY + kPairAddY)
// (factors wrap at 32 bits; the product and the sum at 64).  Unless its first factor
// is zero the term is injective in the second frame, both factors move with the
// position, and it costs one 32 x 32 -> 64-bit multiply-add per two frames; and every
// block but a short path's single one holds 16 frames of the path, so hashing it needs
// no mask.  (A collision costs only time: every table match is verified frame by
// frame.)
constexpr uint32_t kPairMulX = 0x9E3779B9u, kPairMulY = 0x85EBCA6Bu, kPairAddX = 0x27D4EB2Fu,
                   kPairAddY = 0x165667B1u;
__host__ __device__ inline uint64_t pair_term(uint32_t f0, uint32_t f1, uint32_t p) {
  const uint32_t x = f0 + p * kPairMulX + kPairAddX;
  const uint32_t y = f1 + p * kPairMulY + kPairAddY;
  return (uint64_t)x * (uint64_t)y;
}
// first frame of block m of a path of len frames (as above)
__host__ __device__ inline int64_t hash_block_start(int64_t m, int64_t len) {
  const int64_t s = 16 * m;
  return s + 16 > len && len >= 16 ? len - 16 : s;
}
__host__ __device__ inline uint64_t finish_hash(uint64_t s, uint64_t len) {
  uint64_t h = s + len * 0x9E3779B97F4A7C15ull;
  h ^= h >> 33;
  h *= 0xFF51AFD7ED558CCDull;
  h ^= h >> 33;
  h *= 0xC4CEB9FE1A85EC53ull;
  h ^= h >> 33;
  return h;
}

__device__ inline uint32_t hash32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

// ---- arguments -----------------------------------------------------------------------
struct IngestArgs {
  // input batch
  const int64_t *off;
  const uint32_t *fr;
  int64_t n_events, n_frames;
  // unique-path table
  Slot *slot;
  uint64_t cap_mask;
  uint64_t hash_mask;   // all ones, except under a forced-collision test setting
  uint32_t *slot_of;    // [N] output: table slot of every event
  // the tree's path store (for paths seen in earlier calls)
  const uint32_t *pframes;
  const int64_t *pstart;
  const uint32_t *plen;
  // counters [kCtrCount]
  unsigned long long *ctr;
};

// Host-side launch wrappers (one translation unit per kernel family).
void launch_ingest(const IngestArgs &a, int grid, hipStream_t s);
// Sum metrics [N][m] into delta[slot_of[e]][m] (delta starts zeroed).  Every workgroup
// sums its event range into an LDS map keyed by slot; the maps are flushed into
// staging buckets (bucket = slot >> bshift, plain stores, one counter atomic per
// bucket and workgroup), and one workgroup per bucket then adds the bucket's staged
// sums into delta.  Entries that find no room (LDS map full, bucket full) are added
// to delta with atomics.
struct AggStage {
  int32_t bshift;        // bucket of slot s: s >> bshift (agg_bucket_shift(m))
  int64_t nbuckets;      // 0: no staging (maps flushed with atomics)
  int64_t bucket_cap;    // staged entries per bucket
  uint32_t *count;       // [nbuckets], zeroed before the launch
  uint32_t *keys;        // [nbuckets][bucket_cap]
  uint64_t *sums;        // [nbuckets][bucket_cap][m]
};
int agg_bucket_shift(int32_t m);
int64_t agg_max_buckets();
int64_t agg_map_entries(int32_t m);
void launch_aggregate(const uint32_t *slot_of, const uint64_t *w, int64_t n, int32_t m, uint64_t *delta,
                      uint64_t cap, int grid, const AggStage &st, hipStream_t s);
// List the slots claimed in this call (word ref with kEventRef): new_slots, each new
// path's first frame in the batch and length (src_len, two words per path) and padded
// store length (padded, the input of the scan that places the paths in the store), and
// into ctr: kCtrNew (count), kCtrNewFrames (sum of padded store lengths), kCtrNewLen
// (sum of lengths).  new_slots, src_len and padded hold room for every possible new
// path: min(cap, events of the batch).
// part: 2 * collect_blocks(cap) words of scratch.
int64_t collect_blocks(uint64_t cap);
void launch_collect_new(const Slot *slot, uint64_t cap, const int64_t *off, uint32_t *new_slots, int64_t *src_len,
                        uint64_t *padded, unsigned long long *ctr, unsigned long long *part, hipStream_t s);

// Path store: path d occupies frames [pstart[d], pstart[d] + round16(plen[d])) of
// pframes (pstart is a multiple of kStoreAlign, the tail is zero-filled), and its
// checkpoint hashes cp[pstart[d] / kStoreAlign + b] = hash of its prefix of length
// kStoreAlign * (b + 1), for every full block b.
constexpr int kStoreAlign = 16;
__host__ __device__ inline int64_t round_store(int64_t len) {
  return (len + kStoreAlign - 1) / kStoreAlign * kStoreAlign;
}

struct PublishArgs {
  const int64_t *off;        // batch offsets (frames of new paths come from the batch)
  const uint32_t *fr;
  int64_t n_frames;          // frames in the batch
  Slot *slot;
  const uint32_t *new_slots;
  int64_t n_new;
  int64_t d_old;
  uint32_t *pframes;
  uint64_t *pcp;             // checkpoint hashes
  int64_t *pstart;
  uint32_t *plen;
  uint32_t *pslot;
  int64_t store_used;        // frames already used in the store
  const uint64_t *starts;    // [n_new] exclusive prefix sums of the padded lengths
  const int64_t *src_len;    // [n_new][2] first frame in the batch and length of each new path
  uint64_t cp_mask;          // all ones, except under a test setting that forces collisions
};
void launch_publish(const PublishArgs &a, hipStream_t s);
// Exclusive prefix sums of `rows` rows of C uint64 columns (mod 2^64) into out[0..rows),
// totals into out row `rows`; blk holds (rows / 1024 + 1) * C scratch words.
void launch_scan(const uint64_t *in, int64_t rows, int C, uint64_t *blk, uint64_t *out, hipStream_t s);
// sums[d] for d < D after a batch: old paths (d < d_old) add their slot's delta to
// old_sums[d], new ones take it (sums and old_sums are distinct arrays)
void launch_fold_sums(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, const uint64_t *delta,
                      const uint64_t *old_sums, uint64_t *sums, hipStream_t s);
// slot[list[i]] = empty for i < n (the slots published by a call that failed afterwards)
void launch_reset_slots(Slot *slot, const uint32_t *list, int64_t n, hipStream_t s);
void launch_unclaim(Slot *slot, uint64_t cap, hipStream_t s);
void launch_rehash(const uint32_t *pframes, const int64_t *pstart, const uint32_t *plen, int64_t d,
                   Slot *slot, uint64_t cap_mask, uint64_t hash_mask, uint32_t *pslot, hipStream_t s);

struct CanonArgs {
  int64_t d;             // number of distinct full paths
  int64_t id0;           // launch_sort: sorts path ids id0 .. id0 + d - 1 (0 for a full sort)
  const uint32_t *gap;   // launch_sort with gap: orders by (gap[id - id0], path); else nullptr
  int32_t m;
  int32_t exact;         // 1: compare frames only (no checkpoint-hash shortcut)
  const uint32_t *pframes;
  const uint64_t *pcp;
  const int64_t *pstart;
  const uint32_t *plen;
  const uint64_t *psums; // [D][m]
  // outputs / scratch
  uint32_t *order;       // [D] path ids in lexicographic order
  uint32_t *order_tmp;   // [D]
  uint32_t *lcp;         // [D+1] lcp with the previous path in order; lcp[D] = 0
  uint64_t *scan_in;     // [D][1+m] new-node counts and sums in order
  uint64_t *scan_out;    // [D+1][1+m] exclusive prefix sums (+ totals at row D)
  uint64_t *scan_blk;    // block partials
  int64_t scan_blocks;
  uint32_t *sparse;      // [levels][D] range minima of lcp
  int32_t levels;
  uint32_t *chain_parent; // [D]
  uint32_t *win_path;    // [U_max / 64 + 1] path index (in order) holding each 64-node window's first node
  int64_t u_max;
  // node arrays
  uint32_t *parent, *frame, *depth;
  uint32_t *subend;      // [U] end of each node's subtree: its descendants are the ids (u, subend[u])
  uint64_t *excl, *incl;
  unsigned long long *u_out;  // device: [0] node count, [1] order-violation flag
  int grid_nodes;
};
void launch_sort(CanonArgs &a, hipStream_t s);        // leaves the result in a.order
// Order after a merge: every path new in this call (ids d_old .. a.d - 1) finds its
// gap in the previous order (d_old ids, sorted; the old paths keep their relative
// order) by binary search, the new paths are sorted by (gap, path), and both lists
// are placed by integer arithmetic.  scratch: 2 (a.d - d_old) words.  Leaves the
// result in a.order.
void launch_merge_order(CanonArgs &a, const uint32_t *old_order, int64_t d_old, uint32_t *scratch,
                        hipStream_t s);

// Lexicographic order of the D distinct paths through a trie of 16-frame blocks (see
// trie.hip).  Scratch sizes: nblocks = store blocks in use (sum of ceil(len / 16)),
// cap = power of two >= 2 * nblocks.
struct TrieArgs {
  int64_t d;
  int64_t nblocks;
  uint64_t cap;                // node table capacity (power of two)
  const uint32_t *pframes;
  const uint64_t *pcp;
  const int64_t *pstart;
  const uint32_t *plen;
  uint64_t *tkey;              // [cap] node keys (0: empty)
  uint64_t *tinfo;             // [cap] (representative block << 32) | depth
  uint64_t *bpos;              // [nblocks] (path length << 32) | index of the block in its path
  uint32_t *occ;               // [nblocks] node of each store block
  uint32_t *nparent;           // [cap] parent node (cap: the root)
  uint32_t *ncount;            // [cap] distinct paths through the node
  uint32_t *nend;              // [cap + 1] a path ends at the node (cap: the root)
  uint64_t *hist;              // [cap + 1] children per node
  uint64_t *gstart;            // [cap + 2] exclusive prefix sums of hist
  uint32_t *cidx;              // [cap] index of each node among its siblings (root's children:
                               //        (link workgroup << 22) | index within the workgroup)
  uint32_t *rootbase;          // [1024] first index of each link workgroup's root children
  uint32_t *grouped;           // [nblocks] nodes grouped by parent, siblings in order
  uint32_t *grouped2;          // [nblocks] scratch
  uint32_t *posof;             // [cap] position of each node in grouped
  uint64_t *cnt;               // [nblocks] path counts in grouped order
  uint64_t *cnt_scan;          // [nblocks + 1] their exclusive prefix sums
  uint64_t *scan_blk;          // scan scratch: (nblocks / 1024 + 2) words
  uint64_t *lists;             // [4][list_cap] (start << 32 | size): buckets of up to 64, groups of
                               // 65 .. 512 siblings, groups of more than 512, buckets of 65 .. 2048
  int64_t list_cap;
  int64_t large_cap;           // groups of more than 1024 siblings that can be listed
  uint32_t *lgroup;            // [cap + 1] list index of a large group, by parent node
  uint32_t *spl;               // [large_cap][256] splitters (node ids)
  uint32_t *bcnt;              // [large_cap][256] bucket sizes
  unsigned long long *ctr;     // [8]: [0..3] list counts, [kTrieCtrFail] failure
  uint32_t *order;             // [D] out: path ids in lexicographic order
};
constexpr int kTrieCtrFail = 4;
// ctr[kTrieCtrFail] != 0 after the call: the trie could not be used (the caller sorts
// another way).  s2 (may be s): a second stream for the part of the sibling ordering that
// is independent of the large groups, forked from s with `fork` and joined back into s
// with `join` (two events of the caller's, unused when s2 is s).
void launch_trie_sort(const TrieArgs &a, hipStream_t s, hipStream_t s2, hipEvent_t fork, hipEvent_t mid,
                      hipEvent_t join);
void launch_canon(const CanonArgs &a, hipStream_t s);  // lcp, scans, sparse table, emission

struct QueryArgs {
  int64_t q;
  int64_t qn_frames;
  const int64_t *qoff;
  const uint32_t *qfr;
  int64_t d;
  int64_t u;                 // node count (ids are < u)
  int32_t m;
  const uint32_t *pframes;
  const int64_t *pstart;
  const uint32_t *plen;
  const uint32_t *order;
  const uint32_t *lcp;       // [D+1]
  const uint64_t *scan_out;  // column 0 holds the node-id bases
  const uint64_t *excl, *incl;
  int64_t *node_ids;
  uint64_t *qexcl, *qincl;
  unsigned long long *err;
  int64_t *sorted;           // [D][2]: first frame and length of the path at each canonical position
  uint64_t *qtab;            // prefix index [qcap][2] {key, (length << 32) | position}, or null
  uint64_t qcap_mask;
  uint64_t qhash_mask;       // test setting: keys keep only these bits (forced collisions)
};
// the records of `sorted`
void launch_sorted_paths(const QueryArgs &a, hipStream_t s);
// the prefix index of every node (qtab cleared to zero first)
void launch_query_index(const QueryArgs &a, hipStream_t s);
// offsets check of the query batch (err bit 0), run before any output is written
void launch_query_check(const QueryArgs &a, hipStream_t s);
// lookups: through the index when a.qtab is set, else by binary search
void launch_query(const QueryArgs &a, hipStream_t s);

// Correlation-ID join of an activity flush with the registered call paths (activity.hip)
enum : int32_t { kActCtrError = 0, kActCtrUnmatched = 1, kActCtrMin = 2, kActCtrMax = 3, kActCtrCount = 4 };
enum : uint32_t { kActBadOffsets = 1, kActRepeatedId = 2, kActTableFull = 4 };
struct alignas(16) CorrSlot {
  uint64_t key;    // correlation ID (valid once claim != 0)
  uint32_t claim;  // registry index + 1; 0: empty
  uint32_t pad;
};
struct ActivityArgs {
  int64_t n_reg;             // registered paths
  int64_t reg_n_frames;
  const int64_t *reg_off;    // [n_reg + 1]
  const uint64_t *reg_corr;  // [n_reg] correlation IDs
  // dense IDs (max - min < 4 n_reg): a direct table dtab[id - id_min] (registry index + 1,
  // 0: not registered); otherwise the hash table
  bool dense;
  uint64_t id_min, id_span;  // registered IDs lie in [id_min, id_min + id_span]
  uint32_t *dtab;            // [id_span + 1]
  uint64_t cap_mask;         // hash table capacity - 1 (capacity a power of two >= 2 n_reg)
  CorrSlot *table;           // [cap]
  int64_t n_rec;             // activity records
  const uint64_t *rec_corr;  // [n_rec]
  uint32_t *rec_reg;         // [n_rec] registry index of the record's path, kNoSlot if unmatched
  uint32_t *ref;             // [n_reg] 0, or 1 + the index of a record naming the path (its owner)
  unsigned long long *ctr;   // [kActCtrCount]
};
void launch_corr_range(const ActivityArgs &a, hipStream_t s);  // min and max registered ID into ctr
void launch_corr_table(const ActivityArgs &a, hipStream_t s);  // validate offsets, insert, repeated IDs
void launch_corr_join(const ActivityArgs &a, hipStream_t s);
// per-path sums of the matched records; list: scratch of corr_sums_grid(n_rec) stripes
// (n_rec + corr_sums_grid * 256 entries suffice), cnt: [corr_sums_grid(n_rec)]
int64_t corr_sums_grid(int64_t n_rec);
void launch_corr_sums(const ActivityArgs &a, const uint64_t *metrics, int32_t m, uint64_t *sums, uint32_t *list,
                      uint32_t *cnt, hipStream_t s);
void launch_compact_lengths(const ActivityArgs &a, uint64_t *rows, hipStream_t s);
// the batch of referenced paths: offsets [n_paths + 1], frames and metrics; src_start is
// scratch [n_paths]
void launch_compact_gather(const ActivityArgs &a, const uint32_t *reg_frames, const uint64_t *scan,
                           const uint64_t *sums, int32_t m, int64_t n_paths, int64_t n_frames, int64_t *off_out,
                           int64_t *src_start, uint32_t *fr_out, uint64_t *met_out, hipStream_t s);

// Bottom-up view (bottomup.hip): stable radix sort of uint32 (key, value) pairs (four
// passes; hist [256 * radix_blocks(n)], offs [256 * radix_blocks(n) + 1], scan_blk for
// launch_scan over 256 * radix_blocks(n) rows; result back in keys / vals), exclusive
// max-scan of uint64 (blk [maxscan_blocks(n)]), and the view's kernels.
int64_t radix_blocks(int64_t n);
int64_t maxscan_blocks(int64_t n);
void launch_radix_sort(uint32_t *keys, uint32_t *vals, uint32_t *keys_tmp, uint32_t *vals_tmp, int64_t n,
                       uint64_t *hist, uint64_t *offs, uint64_t *scan_blk, hipStream_t s);
void launch_maxscan(const uint64_t *in, int64_t n, uint64_t *blk, uint64_t *out, hipStream_t s);
void launch_bu_keys(const uint32_t *frame, int64_t n, uint32_t *keys, uint32_t *vals, hipStream_t s);
void launch_bu_heads(const uint32_t *K, int64_t n, uint64_t *head, hipStream_t s);
void launch_bu_tag(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint32_t *subend, int64_t n,
                   uint64_t *tag, int64_t *gstart, hipStream_t s);
// slot_ex / slot_in: [n + 1] in node order (the root gets kNoSlot)
void launch_bu_slots(const uint32_t *V, const uint64_t *head, const uint64_t *gscan, const uint64_t *mx, int64_t n,
                     uint32_t *slot_ex, uint32_t *slot_in, hipStream_t s);
void launch_bu_frames(const uint32_t *K, const int64_t *gstart, int64_t G, uint32_t *frames, hipStream_t s);

// Ratio filters over the tree's nodes (filter.hip)
enum : int32_t { kDenOne = 0, kDenMetric = 1, kDenRoot = 2 };
struct FilterArgs {
  int64_t u;
  int32_t m;
  const uint64_t *excl, *incl;  // [U][m]
  const uint32_t *subend;       // [U]
  int32_t num_metric, num_excl;
  int32_t den_kind, den_metric, den_excl;
  int32_t op;                   // +1: ratio above the threshold, -1: below
  uint64_t thr_num, thr_den;
  int32_t leaves_only;
};
constexpr int kFilterTile = 2048;  // nodes per tile of the two passes
int64_t filter_tiles(int64_t u);
// mask [filter_tiles(U) * kFilterTile / 64] (bit per node), count [filter_tiles(U)]
void launch_filter_mask(const FilterArgs &a, uint64_t *mask, uint32_t *count, hipStream_t s);
// pos [tiles + 1]: exclusive scan of count, pos[tiles] = all matches
void launch_filter_scan(const uint32_t *count, int64_t tiles, uint64_t *pos, hipStream_t s);
// writes the first `capacity` matches to out
void launch_filter_write(int64_t u, const uint64_t *mask, const uint64_t *pos, int64_t capacity, int64_t *out,
                         hipStream_t s);
// The filter that allocates nothing keeps its mask, counts and offsets in a static device
// array of kFilterStaticBytes per GPU, enough for kFilterStaticTiles tiles.
constexpr int64_t kFilterStaticTiles = 15360;  // trees of up to 31,457,280 nodes
constexpr size_t kFilterStaticBytes = 4u << 20;
struct FilterScratch {
  uint64_t *mask;   // [tiles * kFilterTile / 64]
  uint32_t *count;  // [tiles]
  uint64_t *pos;    // [tiles + 1]
};
// Device address of the current device's static array (looked up once per device), or
// nullptr if the lookup failed; and the array's parts at that address.
void *filter_static_scratch();
FilterScratch filter_static_layout(void *base);

// Per-path and per-node statistics (stats.hip)
struct StatStage {  // staged per-path statistics of a batch (nbuckets = 0: device atomics instead)
  int32_t bshift;       // bucket of path i: i >> bshift
  int64_t nbuckets;
  int grid;             // workgroups of the per-slot kernel
  int64_t map_entries;  // LDS map entries per workgroup
  uint32_t *ev_path;    // [N] misses (path indices): workgroup g's from its first event index on
  uint64_t *ev_w;       // [N][m]
  uint32_t *map_key;    // [grid][map_entries]
  uint64_t *map_rec;    // [grid][map_entries][1 + 3m]: count, min[m], sq[m][2]
  uint64_t *hist_ev, *hist_map;  // [nbuckets][grid] entries per bucket and workgroup
  uint64_t *off_ev, *off_map;    // their exclusive scans, [nbuckets * grid + 1]
  uint32_t *wg_count;   // [grid][2]: misses, map entries
  uint32_t *st_ev_path;  // bucketed misses [N], values [N][m]
  uint64_t *st_ev_w;
  uint32_t *st_map_key;  // bucketed map entries [grid * map_entries], records
  uint64_t *st_map_rec;
};
struct PathStats {  // kept per path: cnt [D], min [D][m], sq [D][m][2]
  uint64_t *cnt, *min, *sq;
};
struct NodeStatOut {  // any pointer may be null
  uint64_t *count_excl, *count_incl;  // [U]
  uint64_t *min_excl, *min_incl;      // [U][m]
  uint64_t *sumsq_excl, *sumsq_incl;  // [U][m][2]
  double *mean_excl, *mean_incl;      // [U][m]
  double *std_excl, *std_incl;        // [U][m]
};
struct NodeStatArgs {
  int64_t u, d;
  int32_t m;
  const uint64_t *scan_out;  // [d + 1][1 + m] of the canonical emission
  const uint32_t *order;     // [d] canonical position -> path
  const uint64_t *pcnt, *pmin, *psq;
  const uint32_t *subend;         // [u]
  const uint64_t *excl, *incl;    // [u][m]
  uint64_t *rows, *prefix;        // [d][1 + 4m], [d + 1][1 + 4m], canonical path order
  uint32_t *node_path;            // [u]: canonical position of the path that created the node
  uint64_t *cmin, *pre, *suf;     // [d][m]
  uint64_t *tab;                  // [levels][nblk][m], nblk = rmq_blocks(d)
  int64_t nblk;
  int levels;
  NodeStatOut out;
};
int64_t stats_staged_entries(int32_t m);
int stats_bucket_shift(int32_t m);  // largest bucket: 2^shift paths
int64_t stats_max_buckets();
// slot -> path map for paths [0, D); paths [d_old, D) set to no sample
void launch_stats_prepare(int64_t D, int64_t d_old, int32_t m, const uint32_t *pslot, uint32_t *path_of_slot,
                          const PathStats &p, hipStream_t s);
void launch_stats_agg(const uint32_t *slot_of, const uint32_t *path_of_slot, const uint64_t *w, int64_t n, int32_t m,
                      int64_t D, int grid, const PathStats &p, const StatStage &st, uint64_t *scan_blk, hipStream_t s);
int64_t rmq_blocks(int64_t u);
void launch_node_stats(const NodeStatArgs &a, uint64_t *scan_blk, hipStream_t s);

}  // namespace cct
