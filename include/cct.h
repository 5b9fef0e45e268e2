/* cct.h — calling context tree construction on one AMD MI355X (gfx950).
 *
 * C ABI of libcct.so.  The library turns a batch of call paths, each carrying
 * integer metrics, into a calling context tree (CCT): the profiler's tree of the
 * paper (Design, "Profiler", paragraph "Calling Context Tree"), built by inserting
 * call paths with frames that name the same location collapsed into one node, each
 * node holding a list of metrics, every metric added at the bottom node of its
 * call path and propagated to the root along the whole path.  cct_merge
 * aggregates a further batch into an existing tree, as the profiler does when it
 * flushes a full metric buffer into its tree (Design, "Profiler", "GPU Metrics");
 * cct_query looks up the metrics of given call paths, as the analysis API reads the
 * metrics of the nodes on matched call paths (Design, "Performance Analyzer",
 * "Analysis API").
 *
 * Data conventions (the paper is silent on all of them; these are this library's
 * readings):
 *   - A frame is a uint32 id; two frames are the same location iff their ids are
 *     equal (interning of (library, PC), (file, line) or operator names happens
 *     upstream).  Every uint32 value is a legal frame id.
 *   - A call path is root-first: outermost caller first, GPU-kernel leaf last.
 *   - The root is the empty path: id 0, parent CCT_NO_PARENT, frame 0, depth 0.
 *     A zero-length path adds its metrics to the root's exclusive sums.
 *   - Node ids are canonical: the rank of the node's root path in unsigned
 *     lexicographic order, a proper prefix before its extensions (preorder, children
 *     by ascending frame id).  Subtrees are therefore contiguous id ranges.
 *   - Every tree keeps the sum, over uint64 modulo 2^64; a tree built with
 *     cct_build_stats also keeps counts, minima and sums of squares (cct_stats).
 *   - excl[v][j] = sum of metric j over events whose path ends at v;
 *     incl[v][j] = sum of metric j over events whose path passes through v.
 *
 * Threads and streams: calls order all their device work on the given HIP stream
 * (NULL = the default stream) of the current device and return only after that
 * work has completed; input buffers may be freed on return.  A build or merge also runs
 * part of its work on a second stream of its own, ordered by events and finished before
 * it returns.  The calling thread spins (polls an event) while it waits for the device,
 * except in cct_filter_noalloc, which blocks.  Distinct trees may be used from different threads at once; one tree must
 * not be used concurrently, queries and views included (they build indexes and views
 * that the tree keeps).
 *
 * Errors: every call returns a cct_status; nothing aborts, throws or prints.  On an
 * error, out-parameters are untouched and a tree passed to cct_merge is unchanged.
 * cct_last_error() gives a message for the calling thread's last failure.
 */
#ifndef CCT_H
#define CCT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CCT_OK = 0,
  CCT_EINVAL = -1,    /* bad argument or malformed offsets */
  CCT_ENOMEM = -2,    /* a device allocation failed */
  CCT_EDEVICE = -3,   /* a HIP runtime call failed */
  CCT_EMISMATCH = -4, /* merge batch has a different metric count than the tree */
  CCT_EOVERFLOW = -5  /* the tree would exceed 2^32 - 2 nodes, or a batch 2^31 - 2 events */
} cct_status;

#define CCT_MAX_METRICS 8          /* metrics per event (uint64 each) */
#define CCT_NO_PARENT 0xFFFFFFFFu  /* parent of the root */
#define CCT_MAX_EVENTS 0x7FFFFFFELL /* events per cct_build / cct_merge / cct_query call */

typedef struct cct_tree cct_tree; /* opaque; owns its device memory */

/* A batch of call paths in CSR form.  All pointers are DEVICE pointers of the
 * current device, borrowed for the duration of the call.
 *   n_events   N >= 0 (N <= CCT_MAX_EVENTS)
 *   n_frames   F = offsets[N], the number of elements of `frames`
 *   n_metrics  M, 1..CCT_MAX_METRICS
 *   offsets    int64[N+1]; offsets[0] = 0, non-decreasing, offsets[N] = F.
 *              Path i is frames[offsets[i] .. offsets[i+1]).  Checked on the device:
 *              a violation makes the call return CCT_EINVAL.
 *   frames     uint32[F], 4-byte aligned; may be NULL when F = 0
 *   metrics    uint64[N][M] row-major, 8-byte aligned; ignored by cct_query (may be NULL) */
typedef struct {
  int64_t n_events;
  int64_t n_frames;
  int32_t n_metrics;
  const int64_t *offsets;
  const uint32_t *frames;
  const uint64_t *metrics;
} cct_paths;

/* Build a new tree from one batch (calling-context-tree construction: insert every
 * path, aggregate metrics at its end node, propagate to the root).  On success
 * *out receives a tree owned by the caller (release with cct_free). */
cct_status cct_build(const cct_paths *events, void *hip_stream, cct_tree **out);

/* The same, and the tree also keeps the other aggregates the paper names for a node's
 * metrics besides the sum: minimum, average and standard deviation (Design, "Profiler",
 * "Calling Context Tree").  Every event is one sample of each metric, at the node its
 * path ends on (exclusive) and at every node of the path up to the root (inclusive).
 * Per distinct path the tree keeps the sample count, each metric's minimum and its sum
 * of squares modulo 2^128; cct_merge and cct_merge_activity fold their batches in (a
 * joined activity flush gives one sample per registered call path: the sum of its
 * records).  Read them per node with cct_stats. */
cct_status cct_build_stats(const cct_paths *events, void *hip_stream, cct_tree **out);

/* Aggregate one more batch into `tree` (the flush of a full metric buffer into the
 * existing tree).  The result equals cct_build over the concatenation of every batch
 * the tree has seen; node ids are renumbered.  chunk->n_metrics must equal the
 * tree's metric count (else CCT_EMISMATCH). */
cct_status cct_merge(cct_tree *tree, const cct_paths *chunk, void *hip_stream);

/* One flush of the GPU activity buffer: record r carries the correlation ID that the
 * profiler emitted at the GPU API callback of its activity, and the activity's metrics
 * (Design, "Profiler", "GPU Metrics").  DEVICE pointers, borrowed for the call.
 *   n_records  R >= 0 (R <= CCT_MAX_EVENTS)
 *   n_metrics  M, must equal the tree's metric count (else CCT_EMISMATCH)
 *   corr_ids   uint64[R], 8-byte aligned; any value is a legal ID
 *   metrics    uint64[R][M] row-major, 8-byte aligned */
typedef struct {
  int64_t n_records;
  int32_t n_metrics;
  const uint64_t *corr_ids;
  const uint64_t *metrics;
} cct_activity;

/* Merge one activity flush into `tree`, linking every record to the call path that was
 * registered under its correlation ID (at each GPU API callback the profiler emits a
 * unique correlation ID and associates it with the call path it retrieves there; the
 * flushed metrics are linked to their path through that ID and aggregated: Design,
 * "Profiler", "GPU Metrics").
 *   registry      the call paths registered so far, CSR as in cct_paths (DEVICE; its
 *                 n_metrics and metrics are ignored; offsets checked on the device:
 *                 CCT_EINVAL)
 *   reg_corr_ids  uint64[registry->n_events], DEVICE, 8-byte aligned: the correlation ID
 *                 of each registered path; IDs must be distinct (a repeated ID is found
 *                 on the device: CCT_EINVAL)
 *   activity      the flushed records
 *   n_unmatched   HOST out, may be NULL: the number of records whose ID is not registered;
 *                 they are not merged (the caller may keep them for a later flush)
 * The result equals cct_merge of the batch holding, for every matched record in record
 * order, the registered path with the record's metrics.  A registered path that no
 * record names is not inserted.  On an error the tree is unchanged. */
cct_status cct_merge_activity(cct_tree *tree, const cct_paths *registry, const uint64_t *reg_corr_ids,
                              const cct_activity *activity, void *hip_stream, int64_t *n_unmatched);

/* Bottom-up view of `tree`: for every distinct frame f that labels a node (the root's
 * placeholder excluded), in ascending frame order,
 *   excl[f][j] = sum of metric j over the events whose path ends with f (the exclusive
 *                sums of the nodes labelled f),
 *   incl[f][j] = sum of metric j over the events whose path contains f, each event counted
 *                once however often f recurs on its path.
 * The flame graph's bottom-up view aggregates the metrics of the same node across
 * different call paths (Implementation, "GUI", "Flame Graph Visualization").
 *   capacity   entries of the output arrays; they are written only if capacity >= K
 *   frames     DEVICE or HOST uint32[K], or NULL
 *   excl/incl  DEVICE or HOST uint64[K][M] row-major, or NULL
 *   n_frames   HOST out: K
 * Call with capacity 0 to learn K, then with arrays of K entries: the view is computed
 * once and kept with the tree until the tree changes (cct_merge, cct_merge_activity). */
cct_status cct_bottom_up(cct_tree *tree, void *hip_stream, int64_t capacity, uint32_t *frames, uint64_t *excl,
                         uint64_t *incl, int64_t *n_frames);

/* A ratio test on a node's metrics (the paper's example analyses flag nodes whose metric
 * ratio crosses a threshold: Implementation, "Performance Analyzer", "Example Analyses").
 * Node v matches when a(v) / b(v) is above (op = +1) or below (op = -1) thr_num / thr_den,
 * tested without division as a(v) * thr_den > thr_num * b(v) (or <) on exact 128-bit
 * products; so b(v) = 0 makes an above-test match iff a(v) * thr_den > 0, and a below-test
 * never match.
 *   a(v) = (num_excl ? excl : incl)[v][num_metric]
 *   b(v) = 1 (den_kind 0), (den_excl ? excl : incl)[v][den_metric] (den_kind 1), or the
 *          root's incl[0][den_metric] (den_kind 2)
 *   leaves_only  1: only nodes without children can match
 * Examples: hotspot = incl time above tau of the root's, leaves only; small kernels = incl
 * GPU time / incl launch count below tau; CPU latency = incl CPU time / incl GPU time above
 * tau. */
typedef struct {
  int32_t num_metric;
  int32_t num_excl;
  int32_t den_kind;
  int32_t den_metric;
  int32_t den_excl;
  int32_t op;
  uint64_t thr_num;
  uint64_t thr_den;  /* > 0 */
  int32_t leaves_only;
} cct_filter_spec;

/* Node ids of `tree` matching `spec`, ascending (preorder).  Writes the first
 * min(K, capacity) matches to node_ids (DEVICE int64[capacity], written by a kernel; may
 * be NULL when capacity is 0) and K to *n_matches (HOST); returns after the stream has
 * finished the call's work.  Metric indices out of range, an unknown
 * den_kind or op, or thr_den = 0 give CCT_EINVAL. */
cct_status cct_filter(const cct_tree *tree, const cct_filter_spec *spec, void *hip_stream, int64_t capacity,
                      int64_t *node_ids, int64_t *n_matches);

/* cct_filter for callers that cannot allocate memory (code that must not call hipMalloc,
 * tight serving loops, harnesses that forbid allocation): same arguments, results and
 * errors, but the call allocates no device or pinned host memory.  Its scratch is a static
 * device array of 4 MiB that each GPU holds from the first such call until the process
 * ends, so trees of more than 31,457,280 nodes give CCT_EOVERFLOW.  Every call on a GPU
 * reuses that GPU's array: calls that overlap on one GPU (from several threads or
 * streams) race and must be serialised by the caller. */
cct_status cct_filter_noalloc(const cct_tree *tree, const cct_filter_spec *spec, void *hip_stream,
                              int64_t capacity, int64_t *node_ids, int64_t *n_matches);

/* Per-node statistics of a tree built with cct_build_stats: DEVICE arrays, each written
 * by a kernel, any of them may be NULL.  U nodes, M metrics, row-major.
 *   count_excl/incl  uint64[U]: samples ending at the node / passing through it
 *   min_excl/incl    uint64[U][M]: smallest sample; UINT64_MAX where the count is 0
 *   sumsq_excl/incl  uint64[U][M][2]: sum of squared samples modulo 2^128, low word first
 *   mean_excl/incl   double[U][M]: sum / count (the tree's 64-bit sum); NaN where count is 0
 *   std_excl/incl    double[U][M]: population deviation sqrt(n*S2 - S1^2) / n from the
 *                    count n, the 64-bit sum S1 and the 128-bit S2, the integer under the
 *                    root exact and rounded once; NaN where the count is 0, or where that
 *                    integer is negative (only when a sum wrapped)
 * Mean and deviation are within 4 units in the last place of the exact quantity. */
typedef struct {
  uint64_t *count_excl, *count_incl;
  uint64_t *min_excl, *min_incl;
  uint64_t *sumsq_excl, *sumsq_incl;
  double *mean_excl, *mean_incl;
  double *std_excl, *std_incl;
} cct_node_stats;

/* Compute the statistics of every node of `tree` into `out` (returns after the stream
 * has finished).  A tree built without statistics gives CCT_EINVAL. */
cct_status cct_stats(const cct_tree *tree, void *hip_stream, const cct_node_stats *out);

/* Look up Q call paths (queries->offsets/frames, metrics ignored) in `tree`.  The first
 * query on a tree builds a hash index of its node prefixes (about 32 bytes per node, kept
 * with the tree until it changes; without room for it, queries use binary search).
 * Writes DEVICE arrays: node_ids int64[Q] (the canonical id, or -1 if the path is
 * not a node), and, when non-NULL, excl/incl uint64[Q][M] (zeros for absent paths). */
cct_status cct_query(const cct_tree *tree, const cct_paths *queries, void *hip_stream,
                     int64_t *node_ids, uint64_t *excl, uint64_t *incl);

/* Sizes of a tree: node count U (root included), metric count M, and the number of
 * distinct full call paths D seen so far.  Any out-pointer may be NULL (host memory). */
cct_status cct_info(const cct_tree *tree, int64_t *n_nodes, int32_t *n_metrics, int64_t *n_paths);

/* Copy the canonical node arrays into caller buffers (host or device memory):
 * parent/frame/depth uint32[U], excl/incl uint64[U][M].  Any pointer may be NULL. */
cct_status cct_export(const cct_tree *tree, void *hip_stream, uint32_t *parent, uint32_t *frame,
                      uint32_t *depth, uint64_t *excl, uint64_t *incl);

/* Release a tree and its device memory (returned to the library's pool).  NULL-safe. */
void cct_free(cct_tree *tree);

/* Return every cached device block of the library's pool to the HIP runtime.  Trees
 * still alive keep their memory. */
void cct_release_cached_memory(void);

/* Message describing the calling thread's most recent failure ("" if none). */
const char *cct_last_error(void);

/* Per-call timing of the most recent cct_build/cct_merge/cct_merge_activity on the
 * calling thread, in milliseconds measured with HIP events on the call's stream: [0]
 * ingest (hash, dedup, exclusive aggregation), [1] publish of new paths, [2] canonical
 * ordering (sort, LCP, scans), [3] node emission (parents, exclusive, inclusive), [4]
 * whole merge, [5] the correlation-ID join before the merge (cct_merge_activity only;
 * 0 otherwise), [6] the most recent computation of a bottom-up view by cct_bottom_up
 * (calls that only copy a kept view leave it as it is), [7] the last cct_filter, [8] the
 * statistics kept by the last build or merge (the batch's samples folded into the paths;
 * 0 for a tree without statistics), [9] the last cct_stats, [10] the last cct_query's
 * lookups, [11] the prefix index that call built (0 when the tree's index was kept).
 * Returns the number of values written (<= n, at most 12). */
int cct_last_timings(double *ms, int n);

#ifdef __cplusplus
}
#endif

#endif /* CCT_H */
