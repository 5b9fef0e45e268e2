// ORACLE — test infrastructure only.  Only tests/, __graft_entry__.smoke() and the
// bench's cpu_baseline leg may load this library.  It shares no code with the HIP
// path (no headers, helpers, tables or kernels) and never sees its outputs except as
// data handed to or_check.
//
// What it computes: the calling context tree of the paper's profiler (Design,
// "Profiler", paragraph "Calling Context Tree"): call paths are inserted into a tree
// whose nodes merge frames that name one location, each node holds a list
// of metrics, a metric is added at the bottom node of its call path and propagated to
// the root along the whole path.  Frames are uint32 ids (equal iff the ids are equal),
// the sum is the only aggregate, sums wrap modulo 2^64, the root is the empty path,
// and node ids are the rank of a node's root path in unsigned lexicographic order
// (a proper prefix first), i.e. preorder with children visited by ascending frame.
//
// Optionally (or_create_stats) each node also keeps the other aggregates the paper
// names for a node's metrics (same paragraph: sum, minimum, average and standard
// deviation), updated by every event on every node of its path, the root included
// (inclusive), and at the path's end node (exclusive): the sample count, the minimum
// and the sum of squares (exact modulo 2^128).  The mean and the standard deviation are
// derived from these integers by the Python side.
//
// Parity of every function here is pinned by tests against hand-worked trees,
// brute-force prefix enumeration, closed forms and invariants; the paper itself prints
// no tree values, so nothing here is pinned to a printed number.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <thread>
#include <unordered_map>
#include <vector>

namespace {

constexpr uint32_t kNoParent = 0xFFFFFFFFu;

// A plain trie: one std::map of children per node, metrics summed at the node where
// a path ends ("exclusive").
struct Trie {
  struct Node {
    std::map<uint32_t, uint32_t> kids;  // frame -> node index
  };
  int32_t m;
  std::vector<Node> nodes;
  std::vector<uint64_t> excl;  // [node][m]
  // canonical arrays after finalize()
  std::vector<uint32_t> parent, frame, depth;
  std::vector<uint64_t> c_excl, c_incl;
  // statistics (when `stats`), indexed like excl: [node] counts, [node][m] minima and
  // sums of squares; c_* in canonical order after finalize()
  bool stats = false;
  std::vector<uint64_t> ex_cnt, in_cnt, ex_min, in_min;
  std::vector<unsigned __int128> ex_sq, in_sq;
  std::vector<uint64_t> c_ex_cnt, c_in_cnt, c_ex_min, c_in_min;
  std::vector<unsigned __int128> c_ex_sq, c_in_sq;

  explicit Trie(int32_t m_, bool with_stats = false) : m(m_), nodes(1), excl(m_, 0), stats(with_stats) {
    if (stats) add_stat_rows();
  }

  void add_stat_rows() {
    ex_cnt.push_back(0); in_cnt.push_back(0);
    ex_min.insert(ex_min.end(), m, UINT64_MAX); in_min.insert(in_min.end(), m, UINT64_MAX);
    ex_sq.insert(ex_sq.end(), m, 0); in_sq.insert(in_sq.end(), m, 0);
  }

  // one sample per metric at node v: count, minimum, sum of squares
  static void sample(uint64_t &cnt, uint64_t *mn, unsigned __int128 *sq, const uint64_t *w, int32_t m) {
    ++cnt;
    for (int32_t j = 0; j < m; ++j) {
      const uint64_t x = w ? w[j] : 0;
      mn[j] = std::min(mn[j], x);
      sq[j] += (unsigned __int128)x * x;  // wraps mod 2^128
    }
  }

  // Insert one call path and add its metrics at the node it ends on.
  // With statistics, the event is a sample of every node on its path, the root included.
  void insert(const uint32_t *path, int64_t len, const uint64_t *w) {
    uint32_t v = 0;
    if (stats) sample(in_cnt[0], &in_min[0], &in_sq[0], w, m);
    for (int64_t k = 0; k < len; ++k) {
      auto it = nodes[v].kids.find(path[k]);
      if (it == nodes[v].kids.end()) {
        uint32_t c = (uint32_t)nodes.size();
        nodes[v].kids.emplace(path[k], c);
        nodes.emplace_back();
        excl.insert(excl.end(), m, 0);
        if (stats) add_stat_rows();
        v = c;
      } else {
        v = it->second;
      }
      if (stats) sample(in_cnt[v], &in_min[(size_t)v * m], &in_sq[(size_t)v * m], w, m);
    }
    for (int32_t j = 0; j < m; ++j) excl[(size_t)v * m + j] += w ? w[j] : 0;  // wraps mod 2^64
    if (stats) sample(ex_cnt[v], &ex_min[(size_t)v * m], &ex_sq[(size_t)v * m], w, m);
  }

  // Number the nodes in preorder with children in ascending frame order (std::map
  // iterates keys in ascending unsigned order), then propagate every node's metrics to
  // all of its ancestors: inclusive = exclusive + sum of the children's inclusive.
  int64_t finalize() {
    const size_t U = nodes.size();
    parent.assign(U, 0); frame.assign(U, 0); depth.assign(U, 0);
    c_excl.assign(U * m, 0); c_incl.assign(U * m, 0);
    std::vector<uint32_t> id_of(U);
    if (stats) {
      c_ex_cnt.assign(U, 0); c_in_cnt.assign(U, 0);
      c_ex_min.assign(U * m, 0); c_in_min.assign(U * m, 0); c_ex_sq.assign(U * m, 0); c_in_sq.assign(U * m, 0);
    }
    struct Item { uint32_t node, parent_id, frame, depth; };
    std::vector<Item> stack{{0, kNoParent, 0, 0}};
    uint32_t next = 0;
    while (!stack.empty()) {
      Item it = stack.back();
      stack.pop_back();
      uint32_t id = next++;
      id_of[it.node] = id;
      parent[id] = it.parent_id; frame[id] = it.frame; depth[id] = it.depth;
      for (int32_t j = 0; j < m; ++j) c_excl[(size_t)id * m + j] = excl[(size_t)it.node * m + j];
      if (stats) {
        c_ex_cnt[id] = ex_cnt[it.node]; c_in_cnt[id] = in_cnt[it.node];
        for (int32_t j = 0; j < m; ++j) {
          const size_t a = (size_t)id * m + j, b = (size_t)it.node * m + j;
          c_ex_min[a] = ex_min[b]; c_in_min[a] = in_min[b]; c_ex_sq[a] = ex_sq[b]; c_in_sq[a] = in_sq[b];
        }
      }
      // push children in descending frame order so the smallest is visited first
      const auto &kids = nodes[it.node].kids;
      for (auto r = kids.rbegin(); r != kids.rend(); ++r) stack.push_back({r->second, id, r->first, it.depth + 1});
    }
    // post-order accumulation: in preorder every child has a larger id than its parent
    c_incl = c_excl;
    for (size_t v = U; v-- > 1;)
      for (int32_t j = 0; j < m; ++j) c_incl[(size_t)parent[v] * m + j] += c_incl[v * m + j];
    return (int64_t)U;
  }
};

bool valid_offsets(int64_t n, const int64_t *off) {
  if (n < 0 || !off || off[0] != 0) return false;
  for (int64_t i = 0; i < n; ++i) if (off[i + 1] < off[i]) return false;
  return true;
}

}  // namespace

extern "C" {

// ---- std::map trie oracle (incremental: ingest any number of event batches) ----
void *or_create(int32_t n_metrics) {
  if (n_metrics < 1 || n_metrics > 64) return nullptr;
  return new Trie(n_metrics);
}
// The same, keeping per-node statistics (count, minimum, sum of squares).
void *or_create_stats(int32_t n_metrics) {
  if (n_metrics < 1 || n_metrics > 64) return nullptr;
  return new Trie(n_metrics, true);
}
void or_destroy(void *h) { delete static_cast<Trie *>(h); }

// Insert events [0, n) of one CSR batch.  Returns 0, or -1 on malformed offsets.
int or_ingest(void *h, int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics) {
  Trie *t = static_cast<Trie *>(h);
  if (!t || !valid_offsets(n, offsets)) return -1;
  for (int64_t i = 0; i < n; ++i)
    t->insert(frames + offsets[i], offsets[i + 1] - offsets[i], metrics ? metrics + (size_t)i * t->m : nullptr);
  return 0;
}

// Compute the canonical arrays; returns the node count U (root included).
int64_t or_finalize(void *h) { return static_cast<Trie *>(h)->finalize(); }

// Copy canonical arrays out (any pointer may be NULL).  excl/incl are [U][M].
int or_export(void *h, uint32_t *parent, uint32_t *frame, uint32_t *depth, uint64_t *excl, uint64_t *incl) {
  Trie *t = static_cast<Trie *>(h);
  const size_t U = t->parent.size();
  if (parent) std::memcpy(parent, t->parent.data(), U * 4);
  if (frame) std::memcpy(frame, t->frame.data(), U * 4);
  if (depth) std::memcpy(depth, t->depth.data(), U * 4);
  if (excl) std::memcpy(excl, t->c_excl.data(), U * t->m * 8);
  if (incl) std::memcpy(incl, t->c_incl.data(), U * t->m * 8);
  return 0;
}

// Statistics in canonical order after or_finalize (any pointer may be NULL): counts
// [U], minima [U][M] (UINT64_MAX where the count is 0), sums of squares [U][M][2]
// (low word first).  Returns -1 if the oracle keeps no statistics.
int or_stats_export(void *h, uint64_t *ex_cnt, uint64_t *in_cnt, uint64_t *ex_min, uint64_t *in_min,
                    uint64_t *ex_sq, uint64_t *in_sq) {
  Trie *t = static_cast<Trie *>(h);
  if (!t->stats) return -1;
  const size_t U = t->parent.size(), um = U * t->m;
  if (ex_cnt) std::memcpy(ex_cnt, t->c_ex_cnt.data(), U * 8);
  if (in_cnt) std::memcpy(in_cnt, t->c_in_cnt.data(), U * 8);
  if (ex_min) std::memcpy(ex_min, t->c_ex_min.data(), um * 8);
  if (in_min) std::memcpy(in_min, t->c_in_min.data(), um * 8);
  for (size_t i = 0; i < um; ++i) {
    if (ex_sq) { ex_sq[2 * i] = (uint64_t)t->c_ex_sq[i]; ex_sq[2 * i + 1] = (uint64_t)(t->c_ex_sq[i] >> 64); }
    if (in_sq) { in_sq[2 * i] = (uint64_t)t->c_in_sq[i]; in_sq[2 * i + 1] = (uint64_t)(t->c_in_sq[i] >> 64); }
  }
  return 0;
}

// ---- brute force: every prefix of every event into an ordered set of vectors ----
// std::set<std::vector<uint32_t>> orders by std::lexicographical_compare on unsigned
// elements, so iteration order is the node id.  excl/incl by a double loop over
// events x nodes.  O(N * L^2 * log); tiny inputs only.  Call with NULL outputs to get U.
int64_t or_brute(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics,
                 int32_t m, uint32_t *parent, uint32_t *frame, uint32_t *depth, uint64_t *excl,
                 uint64_t *incl) {
  if (!valid_offsets(n, offsets) || m < 1) return -1;
  std::set<std::vector<uint32_t>> prefixes;
  for (int64_t i = 0; i < n; ++i)
    for (int64_t k = 0; k <= offsets[i + 1] - offsets[i]; ++k)
      prefixes.insert(std::vector<uint32_t>(frames + offsets[i], frames + offsets[i] + k));
  prefixes.insert(std::vector<uint32_t>());
  const int64_t U = (int64_t)prefixes.size();
  if (!parent && !frame && !depth && !excl && !incl) return U;
  std::vector<std::vector<uint32_t>> nodes(prefixes.begin(), prefixes.end());
  std::map<std::vector<uint32_t>, uint32_t> id;
  for (int64_t v = 0; v < U; ++v) id[nodes[v]] = (uint32_t)v;
  for (int64_t v = 0; v < U; ++v) {
    const auto &p = nodes[v];
    if (parent) parent[v] = p.empty() ? kNoParent : id[std::vector<uint32_t>(p.begin(), p.end() - 1)];
    if (frame) frame[v] = p.empty() ? 0 : p.back();
    if (depth) depth[v] = (uint32_t)p.size();
    for (int32_t j = 0; j < m; ++j) {
      uint64_t se = 0, si = 0;
      for (int64_t i = 0; i < n; ++i) {
        const int64_t L = offsets[i + 1] - offsets[i];
        const uint32_t *f = frames + offsets[i];
        if ((int64_t)p.size() > L) continue;
        if (!std::equal(p.begin(), p.end(), f)) continue;
        const uint64_t w = metrics[(size_t)i * m + j];
        si += w;
        if ((int64_t)p.size() == L) se += w;
      }
      if (excl) excl[(size_t)v * m + j] = se;
      if (incl) incl[(size_t)v * m + j] = si;
    }
  }
  return U;
}

// ---- point queries: one node's sums by a scan over all events ----
// For each query path q: count = #events whose path has q as a prefix,
// excl[j] = sum of w_j over events whose path equals q, incl[j] = sum over events
// whose path has q as a prefix.  Works at any trace size (O(F) per query); queries
// are spread over `threads` threads.
int or_point_query(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics,
                   int32_t m, int64_t nq, const int64_t *q_offsets, const uint32_t *q_frames,
                   int64_t *count, uint64_t *excl, uint64_t *incl, int threads) {
  if (!valid_offsets(n, offsets) || !valid_offsets(nq, q_offsets) || m < 1) return -1;
  auto work = [&](int64_t qa, int64_t qb) {
    for (int64_t q = qa; q < qb; ++q) {
      const int64_t ql = q_offsets[q + 1] - q_offsets[q];
      const uint32_t *qf = q_frames + q_offsets[q];
      int64_t c = 0;
      std::vector<uint64_t> se(m, 0), si(m, 0);
      for (int64_t i = 0; i < n; ++i) {
        const int64_t L = offsets[i + 1] - offsets[i];
        if (L < ql) continue;
        if (std::memcmp(frames + offsets[i], qf, (size_t)ql * 4) != 0) continue;
        ++c;
        for (int32_t j = 0; j < m; ++j) {
          si[j] += metrics[(size_t)i * m + j];
          if (L == ql) se[j] += metrics[(size_t)i * m + j];
        }
      }
      count[q] = c;
      for (int32_t j = 0; j < m; ++j) { excl[(size_t)q * m + j] = se[j]; incl[(size_t)q * m + j] = si[j]; }
    }
  };
  if (threads < 1) threads = 1;
  std::vector<std::thread> ts;
  int64_t step = (nq + threads - 1) / threads;
  for (int t = 0; t < threads && t * step < nq; ++t)
    ts.emplace_back(work, t * step, std::min(nq, (t + 1) * step));
  for (auto &t : ts) t.join();
  return 0;
}

// ---- invariant checker for any calling context tree in canonical form ----
// Returns 0 if every invariant holds, else a positive code naming the first failure
// (and writes the offending node to *bad):
//  1 root fields (parent sentinel, frame 0, depth 0)     2 parent[v] >= v
//  3 depth[v] != depth[parent[v]] + 1                     4 siblings not strictly
//    increasing in frame as ids increase                  5 ids are not a preorder
//    (the parent of v is not on the current root path)    6 incl != excl + sum of
//    children's incl (mod 2^64)                           7 incl[root] != total
//  8 sum of excl != incl[root]
int or_check(int64_t U, int32_t m, const uint32_t *parent, const uint32_t *frame, const uint32_t *depth,
             const uint64_t *excl, const uint64_t *incl, const uint64_t *total, int64_t *bad) {
  auto fail = [&](int code, int64_t v) { if (bad) *bad = v; return code; };
  if (U < 1) return fail(1, 0);
  if (parent[0] != kNoParent || frame[0] != 0 || depth[0] != 0) return fail(1, 0);
  std::vector<int64_t> last_child(U, -1);
  std::vector<uint32_t> path{0};
  for (int64_t v = 1; v < U; ++v) {
    const uint32_t p = parent[v];
    if (p >= (uint64_t)v) return fail(2, v);
    if (depth[v] != depth[p] + 1) return fail(3, v);
    if (last_child[p] >= 0 && !(frame[last_child[p]] < frame[v])) return fail(4, v);
    last_child[p] = v;
    while (!path.empty() && path.back() != p) path.pop_back();
    if (path.empty()) return fail(5, v);
    path.push_back((uint32_t)v);
  }
  std::vector<uint64_t> acc(excl, excl + (size_t)U * m);
  for (int64_t v = U - 1; v >= 1; --v)
    for (int32_t j = 0; j < m; ++j) acc[(size_t)parent[v] * m + j] += incl[(size_t)v * m + j];
  for (int64_t v = 0; v < U; ++v)
    for (int32_t j = 0; j < m; ++j)
      if (acc[(size_t)v * m + j] != incl[(size_t)v * m + j]) return fail(6, v);
  for (int32_t j = 0; j < m; ++j) {
    if (total && incl[j] != total[j]) return fail(7, 0);
    uint64_t s = 0;
    for (int64_t v = 0; v < U; ++v) s += excl[(size_t)v * m + j];
    if (s != incl[j]) return fail(8, 0);
  }
  return 0;
}

// ---- bottom-up view, from the events (Implementation, "GUI": the bottom-up view
// aggregates the metrics of the same node across different call paths) ----
// For every frame f on some path, ascending: excl[f] = sum of w over the events whose path
// ends with f; incl[f] = sum of w over the events whose path contains f, each event once
// (its distinct frames: a sorted, de-duplicated copy of the path).
struct BottomUp {
  int32_t m;
  std::vector<uint32_t> frames;
  std::vector<uint64_t> excl, incl;
};

// Computes the view into a handle (NULL on malformed offsets); or_bottom_up_fetch copies
// it out (frames ascending), or_bottom_up_free releases it.
void *or_bottom_up(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics, int32_t m) {
  if (!valid_offsets(n, offsets) || m < 1) return nullptr;
  // frame -> row of the accumulators (a hash map: ordered output comes from a final sort)
  std::unordered_map<uint32_t, size_t> row;
  std::vector<uint64_t> ex, in;
  auto row_of = [&](uint32_t f) {
    auto it = row.find(f);
    if (it != row.end()) return it->second;
    const size_t r = row.size();
    row.emplace(f, r);
    ex.resize(ex.size() + m, 0);
    in.resize(in.size() + m, 0);
    return r;
  };
  std::vector<uint32_t> distinct;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t *f = frames + offsets[i];
    const int64_t L = offsets[i + 1] - offsets[i];
    if (L == 0) continue;
    const uint64_t *w = metrics + (size_t)i * m;
    const size_t re = row_of(f[L - 1]);
    for (int32_t j = 0; j < m; ++j) ex[re * m + j] += w[j];
    distinct.assign(f, f + L);
    std::sort(distinct.begin(), distinct.end());
    distinct.erase(std::unique(distinct.begin(), distinct.end()), distinct.end());
    for (uint32_t x : distinct) {
      const size_t r = row_of(x);
      for (int32_t j = 0; j < m; ++j) in[r * m + j] += w[j];
    }
  }
  const int64_t K = (int64_t)row.size();
  std::vector<std::pair<uint32_t, size_t>> order(row.begin(), row.end());
  std::sort(order.begin(), order.end());
  auto *v = new BottomUp{m, std::vector<uint32_t>(K), std::vector<uint64_t>((size_t)K * m),
                         std::vector<uint64_t>((size_t)K * m)};
  for (int64_t k = 0; k < K; ++k) {
    const size_t r = order[k].second;
    v->frames[k] = order[k].first;
    for (int32_t j = 0; j < m; ++j) {
      v->excl[(size_t)k * m + j] = ex[r * m + j];
      v->incl[(size_t)k * m + j] = in[r * m + j];
    }
  }
  return v;
}

int64_t or_bottom_up_size(void *h) { return (int64_t)static_cast<BottomUp *>(h)->frames.size(); }

void or_bottom_up_fetch(void *h, uint32_t *frames_out, uint64_t *excl_out, uint64_t *incl_out) {
  const auto *v = static_cast<BottomUp *>(h);
  std::copy(v->frames.begin(), v->frames.end(), frames_out);
  std::copy(v->excl.begin(), v->excl.end(), excl_out);
  std::copy(v->incl.begin(), v->incl.end(), incl_out);
}

void or_bottom_up_free(void *h) { delete static_cast<BottomUp *>(h); }

}  // extern "C"
