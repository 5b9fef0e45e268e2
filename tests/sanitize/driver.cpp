// Host-side sanitizer driver: links the CPU oracle and the trace generators, built with
// -fsanitize=address,undefined by tests/test_sanitize.py, and exercises every exported
// function on small seeded traces of each generator kind.  The oracle's results are
// cross-checked against its own brute force and invariant checker, so a memory error,
// undefined behaviour or an inconsistency ends the run with a nonzero status.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

extern "C" {
void *tg_create(int kind, int64_t n_events, uint64_t seed, uint64_t seed2, int64_t p0, int64_t p1, int64_t p2,
                int threads);
int64_t tg_n_frames(void *h);
int32_t tg_n_metrics(void *h);
int tg_fill(void *h, int64_t *offsets, uint32_t *frames, uint64_t *metrics, int threads);
void tg_destroy(void *h);

void *or_create(int32_t n_metrics);
void *or_create_stats(int32_t n_metrics);
void or_destroy(void *h);
int or_ingest(void *h, int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics);
int64_t or_finalize(void *h);
int or_export(void *h, uint32_t *parent, uint32_t *frame, uint32_t *depth, uint64_t *excl, uint64_t *incl);
int or_stats_export(void *h, uint64_t *ex_cnt, uint64_t *in_cnt, uint64_t *ex_min, uint64_t *in_min, uint64_t *ex_sq,
                    uint64_t *in_sq);
int64_t or_brute(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics, int32_t m,
                 uint32_t *parent, uint32_t *frame, uint32_t *depth, uint64_t *excl, uint64_t *incl);
int or_point_query(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics, int32_t m,
                   int64_t nq, const int64_t *q_offsets, const uint32_t *q_frames, int64_t *count, uint64_t *excl,
                   uint64_t *incl, int threads);
int or_check(int64_t U, int32_t m, const uint32_t *parent, const uint32_t *frame, const uint32_t *depth,
             const uint64_t *excl, const uint64_t *incl, const uint64_t *total, int64_t *bad);
void *or_bottom_up(int64_t n, const int64_t *offsets, const uint32_t *frames, const uint64_t *metrics, int32_t m);
int64_t or_bottom_up_size(void *h);
void or_bottom_up_fetch(void *h, uint32_t *frames_out, uint64_t *excl_out, uint64_t *incl_out);
void or_bottom_up_free(void *h);
}

namespace {

struct Trace {
  std::vector<int64_t> off;
  std::vector<uint32_t> fr;
  std::vector<uint64_t> w;
  int32_t m = 0;
};

bool make(int kind, int64_t n, uint64_t seed, int64_t p0, int64_t p1, int64_t p2, Trace &t) {
  void *h = tg_create(kind, n, seed, seed + 1000, p0, p1, p2, 3);
  if (!h) return false;
  t.m = tg_n_metrics(h);
  t.off.assign(n + 1, 0);
  t.fr.assign((size_t)tg_n_frames(h) + 1, 0);
  t.w.assign((size_t)n * t.m + 1, 0);
  const int rc = tg_fill(h, t.off.data(), t.fr.data(), t.w.data(), 3);
  tg_destroy(h);
  return rc == 0;
}

struct Tree {
  std::vector<uint32_t> parent, frame, depth;
  std::vector<uint64_t> excl, incl;
};

// the oracle's tree of the trace ingested in `parts` batches (a merge for parts > 1)
bool oracle_tree(const Trace &t, int parts, bool stats, Tree &out) {
  const int64_t n = (int64_t)t.off.size() - 1;
  void *o = stats ? or_create_stats(t.m) : or_create(t.m);
  if (!o) return false;
  for (int p = 0; p < parts; ++p) {
    const int64_t a = n * p / parts, b = n * (p + 1) / parts;
    std::vector<int64_t> off(t.off.begin() + a, t.off.begin() + b + 1);
    const int64_t base = off[0];
    for (auto &x : off) x -= base;
    if (or_ingest(o, b - a, off.data(), t.fr.data() + base, t.w.data() + (size_t)a * t.m) != 0) return false;
  }
  const int64_t U = or_finalize(o);
  out.parent.resize(U); out.frame.resize(U); out.depth.resize(U);
  out.excl.resize((size_t)U * t.m); out.incl.resize((size_t)U * t.m);
  if (or_export(o, out.parent.data(), out.frame.data(), out.depth.data(), out.excl.data(), out.incl.data()) != 0)
    return false;
  if (stats) {
    std::vector<uint64_t> c1(U), c2(U), m1((size_t)U * t.m), m2((size_t)U * t.m), s1((size_t)U * t.m * 2),
        s2((size_t)U * t.m * 2);
    if (or_stats_export(o, c1.data(), c2.data(), m1.data(), m2.data(), s1.data(), s2.data()) != 0) return false;
    if (c2[0] != (uint64_t)n) return false;  // every event passes through the root
  }
  or_destroy(o);
  return true;
}

int fail(const char *what, int kind, int64_t n) {
  std::printf("FAIL %s (kind %d, %lld events)\n", what, kind, (long long)n);
  return 1;
}

int run_case(int kind, int64_t n, uint64_t seed, int64_t p0, int64_t p1, int64_t p2, bool brute) {
  Trace t;
  if (!make(kind, n, seed, p0, p1, p2, t)) return fail("generate", kind, n);
  Tree a, b;
  if (!oracle_tree(t, 1, false, a)) return fail("oracle", kind, n);
  if (!oracle_tree(t, 3, true, b)) return fail("oracle in three batches", kind, n);
  if (a.parent != b.parent || a.frame != b.frame || a.depth != b.depth || a.excl != b.excl || a.incl != b.incl)
    return fail("merge differs from one batch", kind, n);
  const int64_t U = (int64_t)a.parent.size();
  std::vector<uint64_t> total(t.m, 0);
  for (int64_t i = 0; i < n; ++i)
    for (int32_t j = 0; j < t.m; ++j) total[j] += t.w[(size_t)i * t.m + j];
  int64_t bad = -1;
  if (or_check(U, t.m, a.parent.data(), a.frame.data(), a.depth.data(), a.excl.data(), a.incl.data(), total.data(),
               &bad) != 0)
    return fail("invariants", kind, n);
  if (brute) {
    Tree c;
    const int64_t Ub = or_brute(n, t.off.data(), t.fr.data(), t.w.data(), t.m, nullptr, nullptr, nullptr, nullptr,
                                nullptr);
    if (Ub != U) return fail("brute-force node count", kind, n);
    c.parent.resize(U); c.frame.resize(U); c.depth.resize(U);
    c.excl.resize((size_t)U * t.m); c.incl.resize((size_t)U * t.m);
    or_brute(n, t.off.data(), t.fr.data(), t.w.data(), t.m, c.parent.data(), c.frame.data(), c.depth.data(),
             c.excl.data(), c.incl.data());
    if (a.parent != c.parent || a.frame != c.frame || a.depth != c.depth || a.excl != c.excl || a.incl != c.incl)
      return fail("brute force", kind, n);
  }
  // point queries of the first paths: the count of each must be at least one
  const int64_t nq = n < 16 ? n : 16;
  std::vector<int64_t> cnt(nq + 1);
  std::vector<uint64_t> qe((size_t)nq * t.m + 1), qi((size_t)nq * t.m + 1);
  if (nq > 0 && or_point_query(n, t.off.data(), t.fr.data(), t.w.data(), t.m, nq, t.off.data(), t.fr.data(),
                               cnt.data(), qe.data(), qi.data(), 2) != 0)
    return fail("point query", kind, n);
  for (int64_t q = 0; q < nq; ++q)
    if (cnt[q] < 1) return fail("point query count", kind, n);
  void *bu = or_bottom_up(n, t.off.data(), t.fr.data(), t.w.data(), t.m);
  if (!bu) return fail("bottom-up view", kind, n);
  const int64_t K = or_bottom_up_size(bu);
  std::vector<uint32_t> bf(K + 1);
  std::vector<uint64_t> be((size_t)K * t.m + 1), bi((size_t)K * t.m + 1);
  or_bottom_up_fetch(bu, bf.data(), be.data(), bi.data());
  or_bottom_up_free(bu);
  for (int64_t k = 1; k < K; ++k)
    if (bf[k - 1] >= bf[k]) return fail("bottom-up frames not ascending", kind, n);
  return 0;
}

}  // namespace

int main() {
  int bad = 0;
  // the named generators at small sizes (kind 4 needs a chunk index in p0)
  bad |= run_case(0, 3000, 11, 0, 0, 0, false);
  bad |= run_case(1, 4000, 12, 0, 0, 0, false);
  bad |= run_case(2, 4000, 13, 0, 0, 0, false);
  bad |= run_case(3, 3000, 14, 0, 0, 0, false);
  bad |= run_case(4, 3000, 15, 7, 0, 0, false);
  bad |= run_case(5, 300, 16, 0, 0, 0, false);
  // tiny random traces over special ids, checked against the brute force
  for (uint64_t s = 0; s < 20; ++s) bad |= run_case(6, 40, 100 + s, 1 + (int64_t)(s % 16), 8, 1 + (int64_t)(s % 8), true);
  for (uint64_t s = 0; s < 5; ++s) bad |= run_case(7, 200, 200 + s, 30, 12, 3, true);
  // malformed offsets are refused, not read past
  std::vector<int64_t> off = {0, 5, 3};
  std::vector<uint32_t> fr(8, 1);
  std::vector<uint64_t> w(2, 1);
  void *o = or_create(1);
  if (or_ingest(o, 2, off.data(), fr.data(), w.data()) == 0) bad |= fail("malformed offsets accepted", -1, 2);
  or_destroy(o);
  std::printf(bad ? "sanitizer driver: FAILED\n" : "sanitizer driver: ok\n");
  return bad;
}
