// Seeded synthetic call-path traces (CSR: offsets int64[N+1], frames uint32[F],
// metrics uint64[N][M]).  Shared by the CPU oracle tests and the GPU path tests;
// holds none of the calling-context-tree arithmetic, only the workload recipes.
//
// The paper builds its calling context tree from call paths that run from Python
// frames through framework operators and C/C++ frames down to a GPU-kernel leaf
// (Design, "Call Path Integration"), profiled on many-small-kernel training
// workloads (Evaluation, "Workloads").  The recipes below reproduce that shape;
// no real profile exists, so every input is synthetic.
//
// Randomness is counter based: every draw is splitmix64 (Steele, Lea, Flood,
// OOPSLA 2014) applied to (seed, stream, index), so each event is reproducible on
// its own and the output does not depend on the thread count.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <unordered_set>
#include <vector>

namespace {

inline uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
inline uint64_t draw(uint64_t seed, uint64_t stream, uint64_t idx) {
  return mix64(mix64(seed ^ mix64(stream * 0xD1B54A32D192ED03ull)) + idx);
}
// uniform integer in [lo, hi] (inclusive), via the high half of a 128-bit product
inline uint64_t uni(uint64_t r, uint64_t lo, uint64_t hi) {
  uint64_t span = hi - lo + 1;
  if (span == 0) return r;  // full 64-bit range
  return lo + (uint64_t)(((__uint128_t)r * span) >> 64);
}
inline double unit(uint64_t r) { return (double)(r >> 11) * (1.0 / 9007199254740992.0); }

enum Stream : uint64_t {
  S_POOL = 1, S_TREE, S_TPL_DEPTH, S_TPL_PARENT, S_TPL_SPLIT, S_TPL_FW, S_TPL_FRAME,
  S_EV_PICK, S_EV_POOL, S_EV_METRIC, S_PERM, S_EV_LEN, S_EV_FRAME, S_DEEP
};

// Zipf(s) over ranks 0..n-1 by inverse CDF on a cumulative weight table.
struct Zipf {
  std::vector<double> cdf;
  Zipf() {}
  Zipf(size_t n, double s) : cdf(n) {
    double acc = 0;
    for (size_t i = 0; i < n; ++i) { acc += std::pow((double)(i + 1), -s); cdf[i] = acc; }
  }
  size_t sample(double u) const {
    double x = u * cdf.back();
    size_t r = std::upper_bound(cdf.begin(), cdf.end(), x) - cdf.begin();
    return r < cdf.size() ? r : cdf.size() - 1;
  }
};

// Seeded permutation of 0..n-1 (Fisher-Yates with counter-based draws).
std::vector<uint32_t> permutation(size_t n, uint64_t seed, uint64_t stream) {
  std::vector<uint32_t> p(n);
  for (size_t i = 0; i < n; ++i) p[i] = (uint32_t)i;
  for (size_t i = n; i > 1; --i) {
    size_t j = uni(draw(seed, stream, i), 0, i - 1);
    std::swap(p[i - 1], p[j]);
  }
  return p;
}

// n distinct frame ids drawn from the full uint32 range; 0 and 0xFFFFFFFF always
// included (ids 0 and 1 of the pool).
std::vector<uint32_t> frame_pool(size_t n, uint64_t seed) {
  std::vector<uint32_t> ids;
  ids.reserve(n);
  std::unordered_set<uint32_t> seen;
  seen.reserve(n * 2);
  ids.push_back(0u); seen.insert(0u);
  if (n > 1) { ids.push_back(0xFFFFFFFFu); seen.insert(0xFFFFFFFFu); }
  for (uint64_t k = 0; ids.size() < n; ++k) {
    uint32_t v = (uint32_t)(draw(seed, S_POOL, k) >> 32);
    if (seen.insert(v).second) ids.push_back(v);
  }
  // shuffle so the two extreme ids land anywhere in the pool's layer ranges
  auto p = permutation(ids.size(), seed, S_POOL + 100);
  std::vector<uint32_t> out(ids.size());
  for (size_t i = 0; i < ids.size(); ++i) out[i] = ids[p[i]];
  return out;
}

template <class F>
void parallel_for(int64_t n, int threads, F f) {
  if (threads <= 1 || n < 4096) { f(0, n); return; }
  std::vector<std::thread> ts;
  int64_t step = (n + threads - 1) / threads;
  for (int t = 0; t < threads; ++t) {
    int64_t a = t * step, b = std::min(n, a + step);
    if (a >= b) break;
    ts.emplace_back([=] { f(a, b); });
  }
  for (auto &t : ts) t.join();
}

// Flat set of template paths.
struct Templates {
  std::vector<int64_t> off{0};
  std::vector<uint32_t> fr;
  std::vector<uint32_t> root;  // index of the root template each one descends from
  size_t size() const { return off.size() - 1; }
  uint32_t len(size_t t) const { return (uint32_t)(off[t + 1] - off[t]); }
};

// Layered program: Python frames, then framework operators, then C/C++ frames, with
// a GPU-kernel leaf last.  Template j < n_roots is fresh; every later template
// branches off a uniformly chosen earlier one at a split depth of
// d - (1 + Geometric(mean 8)), clamped to [1, len(parent)], so it shares at least the
// top-level frame and usually a long prefix with its parent.
struct LayerSpec {
  size_t n_templates, n_roots;
  uint32_t dmin, dmax;
  size_t py, fw, cpp, kern;  // id counts per layer
};

Templates make_layered(const LayerSpec &L, uint64_t seed) {
  size_t total = L.py + L.fw + L.cpp + L.kern;
  std::vector<uint32_t> pool = frame_pool(total, seed);
  const uint32_t *layer_base[4] = {pool.data(), pool.data() + L.py, pool.data() + L.py + L.fw,
                                   pool.data() + L.py + L.fw + L.cpp};
  const size_t layer_n[4] = {L.py, L.fw, L.cpp, L.kern};
  Templates T;
  T.fr.reserve(L.n_templates * (L.dmin + L.dmax) / 2);
  T.root.reserve(L.n_templates);
  const double lq = std::log(1.0 - 1.0 / 8.0);
  for (size_t j = 0; j < L.n_templates; ++j) {
    uint32_t d = (uint32_t)uni(draw(seed, S_TPL_DEPTH, j), L.dmin, L.dmax);
    uint32_t nfw = (uint32_t)uni(draw(seed, S_TPL_FW, j), 1, 4);
    uint32_t P = std::min<uint32_t>(20, d >= 2 ? d - 2 : 0);
    uint32_t fw_end = std::min<uint32_t>(P + nfw, d - 1);
    uint32_t s = 0;
    size_t parent = j;
    if (j >= L.n_roots) {
      parent = uni(draw(seed, S_TPL_PARENT, j), 0, j - 1);
      double u = unit(draw(seed, S_TPL_SPLIT, j));
      uint32_t g = 1 + (uint32_t)std::floor(std::log(1.0 - u) / lq);
      int64_t sp = (int64_t)d - (int64_t)(1 + g);
      sp = std::max<int64_t>(1, std::min<int64_t>(sp, T.len(parent)));
      s = (uint32_t)std::min<int64_t>(sp, d - 1);
      if (s < 1) s = 1;
    }
    size_t beg = T.fr.size();
    for (uint32_t l = 0; l < s; ++l) T.fr.push_back(T.fr[T.off[parent] + l]);
    for (uint32_t l = s; l < d; ++l) {
      int layer = l < P ? 0 : l < fw_end ? 1 : l + 1 < d ? 2 : 3;
      uint64_t r = draw(seed, S_TPL_FRAME, (uint64_t)j * 1024 + l);
      T.fr.push_back(layer_base[layer][uni(r, 0, layer_n[layer] - 1)]);
    }
    (void)beg;
    T.off.push_back((int64_t)T.fr.size());
    T.root.push_back(j < L.n_roots ? (uint32_t)j : T.root[parent]);
  }
  return T;
}

struct Trace {
  int kind = -1;
  int64_t n = 0;
  int32_t m = 1;
  uint64_t seed = 0, seed2 = 0;
  int64_t p0 = 0, p1 = 0, p2 = 0;
  Templates T;
  std::vector<uint32_t> ev_tpl;   // template (or packed recipe) per event
  std::vector<int64_t> offsets;
  // deep-recursion recipe
  std::vector<uint32_t> deep_pool, cycle, entry, tails;
};

// ---------------------------------------------------------------- recipes
// kind 0  tiny: random recursive call-site tree (6,000 sites, 2,000 labels,
//         branching <= 6, depth <= 16); event = root-to-site walk, site ~ Zipf(1.1).
// kind 1  layered, 65,536 templates, depth 8..64, 50,000 ids; template ~ Zipf(1.2).
// kind 2  layered, 262,144 templates, depth 16..128, 200,000 ids; 90% of events from
//         the descendants of 8 "training-loop" roots (each pool Zipf(1.1)).
// kind 3  incremental-merge base: kind-2 program, Zipf(1.1) over its first 60%.
// kind 4  incremental-merge chunk p0 of 32: 80% Zipf(1.1) over templates emitted
//         so far, 20% uniform over the next unseen slice; events from seed p1.
// kind 5  deep recursion: 4 entry frames + a 12-frame cycle to depth d-k,
//         d ~ U{256..512}, then k ~ U{1..8} frames of one of 64 exit tails;
//         1% of events are a single frame.
// kind 6  random small: alphabet p0 (<= 16 special ids), length U{0..p1}, p2
//         metrics drawn from the full uint64 range (exercises wrap-around).
// kind 7  random paths over a p0-id pool, length U{1..p1}, p2 metrics in [0, 2^20).
constexpr uint32_t kSpecial[16] = {0u, 1u, 2u, 0x7FFFFFFFu, 0x80000000u, 0xFFFFFFFFu, 3u, 0xFFFFFFFEu,
                                   0x80000001u, 17u, 0x12345678u, 0xDEADBEEFu, 5u, 0x7FFFFFFEu, 4u, 0xC0000000u};

LayerSpec spec_layered_1m() { return {65536, 64, 8, 64, 20000, 5000, 20000, 5000}; }
LayerSpec spec_layered_16m() { return {262144, 64, 16, 128, 80000, 20000, 80000, 20000}; }

void build_events(Trace &tr, int threads) {
  const int64_t n = tr.n;
  tr.ev_tpl.assign(n, 0);
  std::vector<uint32_t> lens(n);
  const uint64_t seed = tr.seed;
  switch (tr.kind) {
    case 0: {
      // call-site tree
      const size_t n_sites = 6000, n_labels = 2000;
      std::vector<uint32_t> labels = frame_pool(n_labels, seed);
      std::vector<int32_t> parent{-1};
      std::vector<uint32_t> depth{0}, kids{0}, lab{0};
      std::vector<uint32_t> eligible{0};
      std::vector<int32_t> pos_in_elig{0};
      for (uint64_t k = 0; parent.size() < n_sites + 1; ++k) {
        size_t pick = uni(draw(seed, S_TREE, 2 * k), 0, eligible.size() - 1);
        uint32_t p = eligible[pick];
        uint32_t c = (uint32_t)parent.size();
        parent.push_back((int32_t)p);
        depth.push_back(depth[p] + 1);
        kids.push_back(0);
        lab.push_back(labels[uni(draw(seed, S_TREE, 2 * k + 1), 0, n_labels - 1)]);
        pos_in_elig.push_back(-1);
        if (depth[c] < 16) { pos_in_elig[c] = (int32_t)eligible.size(); eligible.push_back(c); }
        if (++kids[p] >= 6) {  // remove p from eligible (swap-pop)
          int32_t at = pos_in_elig[p];
          uint32_t last = eligible.back();
          eligible[at] = last; pos_in_elig[last] = at;
          eligible.pop_back(); pos_in_elig[p] = -1;
        }
      }
      // each site's root-to-site label path becomes a template
      Templates &T = tr.T;
      for (size_t s = 1; s < parent.size(); ++s) {
        std::vector<uint32_t> path;
        for (int32_t v = (int32_t)s; v > 0; v = parent[v]) path.push_back(lab[v]);
        std::reverse(path.begin(), path.end());
        T.fr.insert(T.fr.end(), path.begin(), path.end());
        T.off.push_back((int64_t)T.fr.size());
        T.root.push_back(0);
      }
      Zipf z(T.size(), 1.1);
      auto perm = permutation(T.size(), seed, S_PERM);
      parallel_for(n, threads, [&](int64_t a, int64_t b) {
        for (int64_t i = a; i < b; ++i) {
          uint32_t t = perm[z.sample(unit(draw(seed, S_EV_PICK, i)))];
          tr.ev_tpl[i] = t; lens[i] = T.len(t);
        }
      });
      break;
    }
    case 1: {
      tr.T = make_layered(spec_layered_1m(), seed);
      Zipf z(tr.T.size(), 1.2);
      auto perm = permutation(tr.T.size(), seed, S_PERM);
      parallel_for(n, threads, [&](int64_t a, int64_t b) {
        for (int64_t i = a; i < b; ++i) {
          uint32_t t = perm[z.sample(unit(draw(seed, S_EV_PICK, i)))];
          tr.ev_tpl[i] = t; lens[i] = tr.T.len(t);
        }
      });
      break;
    }
    case 2: {
      tr.T = make_layered(spec_layered_16m(), seed);
      std::vector<uint32_t> hot, cold;
      for (size_t t = 0; t < tr.T.size(); ++t) (tr.T.root[t] < 8 ? hot : cold).push_back((uint32_t)t);
      auto ph = permutation(hot.size(), seed, S_PERM), pc = permutation(cold.size(), seed, S_PERM + 1);
      Zipf zh(hot.size(), 1.1), zc(cold.size(), 1.1);
      parallel_for(n, threads, [&](int64_t a, int64_t b) {
        for (int64_t i = a; i < b; ++i) {
          bool is_hot = unit(draw(seed, S_EV_POOL, i)) < 0.9;
          double u = unit(draw(seed, S_EV_PICK, i));
          uint32_t t = is_hot ? hot[ph[zh.sample(u)]] : cold[pc[zc.sample(u)]];
          tr.ev_tpl[i] = t; lens[i] = tr.T.len(t);
        }
      });
      break;
    }
    case 3:
    case 4: {
      tr.T = make_layered(spec_layered_16m(), seed);  // program from seed A
      const size_t T = tr.T.size();
      const size_t base_n = (T * 6) / 10, slice = (T - base_n) / 32;
      if (tr.kind == 3) {
        Zipf z(base_n, 1.1);
        parallel_for(n, threads, [&](int64_t a, int64_t b) {
          for (int64_t i = a; i < b; ++i) {
            uint32_t t = (uint32_t)z.sample(unit(draw(seed, S_EV_PICK, i)));
            tr.ev_tpl[i] = t; lens[i] = tr.T.len(t);
          }
        });
      } else {
        const int64_t c = tr.p0;
        const uint64_t eseed = tr.seed2 + (uint64_t)c;  // chunk c draws from stream B + c
        const size_t seen = base_n + (size_t)c * slice;
        Zipf z(seen, 1.1);
        parallel_for(n, threads, [&](int64_t a, int64_t b) {
          for (int64_t i = a; i < b; ++i) {
            bool fresh = unit(draw(eseed, S_EV_POOL, i)) < 0.2;
            uint64_t r = draw(eseed, S_EV_PICK, i);
            uint32_t t = fresh ? (uint32_t)(seen + uni(r, 0, slice - 1)) : (uint32_t)z.sample(unit(r));
            tr.ev_tpl[i] = t; lens[i] = tr.T.len(t);
          }
        });
      }
      break;
    }
    case 5: {
      tr.deep_pool = frame_pool(20000, seed);
      tr.cycle.assign(tr.deep_pool.begin(), tr.deep_pool.begin() + 12);
      tr.entry.assign(tr.deep_pool.begin() + 12, tr.deep_pool.begin() + 16);
      tr.tails.resize(64 * 8);
      for (size_t k = 0; k < tr.tails.size(); ++k)
        tr.tails[k] = tr.deep_pool[uni(draw(seed, S_DEEP, k), 0, tr.deep_pool.size() - 1)];
      parallel_for(n, threads, [&](int64_t a, int64_t b) {
        for (int64_t i = a; i < b; ++i) {
          uint64_t r0 = draw(seed, S_EV_POOL, i), r1 = draw(seed, S_EV_PICK, i);
          if (unit(r0) < 0.01) {  // single frame; packed as d = 1
            uint32_t f = (uint32_t)uni(r1, 0, tr.deep_pool.size() - 1);
            tr.ev_tpl[i] = (f << 1) | 1u; lens[i] = 1;
          } else {
            uint32_t d = (uint32_t)uni(r1, 256, 512);
            uint32_t k = (uint32_t)uni(draw(seed, S_EV_LEN, i), 1, 8);
            uint32_t tt = (uint32_t)uni(draw(seed, S_DEEP + 1, i), 0, 63);
            tr.ev_tpl[i] = (d << 11) | (k << 7) | (tt << 1);  // bit 0 clear
            lens[i] = d;
          }
        }
      });
      break;
    }
    case 6:
    case 7: {
      const uint32_t lmax = (uint32_t)tr.p1;
      const bool small = tr.kind == 6;
      parallel_for(n, threads, [&](int64_t a, int64_t b) {
        for (int64_t i = a; i < b; ++i)
          lens[i] = (uint32_t)uni(draw(seed, S_EV_LEN, i), small ? 0 : 1, lmax);
      });
      if (!small) tr.deep_pool = frame_pool((size_t)tr.p0, seed);
      break;
    }
  }
  tr.offsets.assign(n + 1, 0);
  for (int64_t i = 0; i < n; ++i) tr.offsets[i + 1] = tr.offsets[i] + lens[i];
}

void fill(const Trace &tr, int64_t *offsets, uint32_t *frames, uint64_t *metrics, int threads) {
  const int64_t n = tr.n;
  const int32_t m = tr.m;
  std::memcpy(offsets, tr.offsets.data(), sizeof(int64_t) * (n + 1));
  const uint64_t seed = tr.kind == 4 ? tr.seed2 + (uint64_t)tr.p0 : tr.seed;
  parallel_for(n, threads, [&](int64_t a, int64_t b) {
    for (int64_t i = a; i < b; ++i) {
      uint32_t *dst = frames + tr.offsets[i];
      const uint32_t len = (uint32_t)(tr.offsets[i + 1] - tr.offsets[i]);
      switch (tr.kind) {
        case 5:
          if (tr.ev_tpl[i] & 1u) dst[0] = tr.deep_pool[tr.ev_tpl[i] >> 1];
          break;  // deep paths are written below
        case 6:
          for (uint32_t l = 0; l < len; ++l)
            dst[l] = kSpecial[uni(draw(seed, S_EV_FRAME, (uint64_t)i * 4096 + l), 0, (uint64_t)tr.p0 - 1)];
          break;
        case 7:
          for (uint32_t l = 0; l < len; ++l)
            dst[l] = tr.deep_pool[uni(draw(seed, S_EV_FRAME, (uint64_t)i * 4096 + l), 0, tr.deep_pool.size() - 1)];
          break;
        default:
          std::memcpy(dst, tr.T.fr.data() + tr.T.off[tr.ev_tpl[i]], sizeof(uint32_t) * len);
      }
      if (metrics) {
        uint64_t *w = metrics + (size_t)i * m;
        for (int32_t k = 0; k < m; ++k) {
          uint64_t r = draw(seed, S_EV_METRIC, (uint64_t)i * 8 + k);
          uint64_t v;
          switch (tr.kind) {
            case 0: case 5: v = uni(r, 1000, 1000000); break;                       // time ns
            case 1: v = k == 0 ? uni(r, 1000, 1000000) : k == 1 ? 1 : uni(r, 0, 1ull << 26); break;
            case 2: v = k == 0 ? uni(r, 1000, 1000000) : uni(r, 0, 1ull << 26); break;
            case 3: case 4:
              v = k == 0 ? uni(r, 1000, 1000000) : k == 1 ? 1 : k == 2 ? uni(r, 0, 1ull << 26) : r;
              break;
            case 6: v = r; break;                                                   // full range
            default: v = uni(r, 0, (1ull << 20) - 1);
          }
          w[k] = v;
        }
      }
    }
  });
  if (tr.kind == 5) {
    // deep-recursion paths are written from their packed recipe
    parallel_for(n, threads, [&](int64_t a, int64_t b) {
      for (int64_t i = a; i < b; ++i) {
        uint32_t code = tr.ev_tpl[i];
        if (code & 1u) continue;
        uint32_t *dst = frames + tr.offsets[i];
        uint32_t d = code >> 11, k = (code >> 7) & 15u, tt = (code >> 1) & 63u;
        uint32_t e = d - k, l = 0;
        for (; l < 4 && l < e; ++l) dst[l] = tr.entry[l];
        for (; l < e; ++l) dst[l] = tr.cycle[(l - 4) % 12];
        for (uint32_t q = 0; q < k; ++q) dst[e + q] = tr.tails[tt * 8 + q];
      }
    });
  }
}

}  // namespace

extern "C" {

// Create a trace recipe.  Returns NULL on bad arguments.
void *tg_create(int kind, int64_t n_events, uint64_t seed, uint64_t seed2, int64_t p0, int64_t p1,
                int64_t p2, int threads) {
  if (kind < 0 || kind > 7 || n_events < 0) return nullptr;
  if ((kind == 6 && (p0 < 1 || p0 > 16 || p1 < 0 || p1 > 4095 || p2 < 1 || p2 > 8)) ||
      (kind == 7 && (p0 < 1 || p1 < 1 || p1 > 4095 || p2 < 1 || p2 > 8)) ||
      (kind == 4 && (p0 < 0 || p0 >= 32)))
    return nullptr;
  Trace *tr = new Trace;
  tr->kind = kind; tr->n = n_events; tr->seed = seed; tr->seed2 = seed2;
  tr->p0 = p0; tr->p1 = p1; tr->p2 = p2;
  static const int32_t mm[6] = {1, 3, 2, 4, 4, 1};
  tr->m = kind <= 5 ? mm[kind] : (int32_t)p2;
  build_events(*tr, threads);
  return tr;
}
int64_t tg_n_frames(void *h) { return static_cast<Trace *>(h)->offsets.back(); }
int32_t tg_n_metrics(void *h) { return static_cast<Trace *>(h)->m; }
// Write the trace into caller buffers of sizes [N+1], [F], [N*M] (metrics may be NULL).
int tg_fill(void *h, int64_t *offsets, uint32_t *frames, uint64_t *metrics, int threads) {
  if (!h || !offsets || !frames) return -1;
  fill(*static_cast<Trace *>(h), offsets, frames, metrics, threads);
  return 0;
}
void tg_destroy(void *h) { delete static_cast<Trace *>(h); }

}  // extern "C"
