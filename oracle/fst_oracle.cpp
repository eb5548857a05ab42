// Reference oracle for reachable-state weighted FST composition.
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
// the CPU-baseline leg of the benchmark may load this library.  It shares no
// code, header, table or helper with the HIP implementation.
//
// What it computes (Argueta & Chiang, "Composing Finite State Transducers on
// GPUs"):
//   * Composition (§2): for M1 = (Q1, Sigma, Gamma, s1, F1, delta1) and
//     M2 = (Q2, Gamma, Delta, s2, F2, delta2), every pair of arcs
//     q1 -a:b/p1-> r1 and q2 -b:c/p2-> r2 sharing the inner symbol b gives a
//     composed arc q1q2 -a:c/p1*p2-> r1r2, and composed arcs that agree in
//     source, target, input and output are merged by adding their weights.
//     The displayed sum in §2 has its bound variable and the output symbol
//     swapped; it is read as delta(q1q2, a, c, r1r2) =
//     sum over b of delta1(q1, a, b, r1) * delta2(q2, b, c, r2), which is what
//     the arc rule just below it states.
//   * Reachable states only (§3.1, §3.2 Algorithm 1): a breadth-first search
//     from s1s2 with a FIFO frontier A and a visited set Q; a popped pair is
//     expanded by joining all its M1 arcs with all its M2 arcs on the inner
//     symbol, and each target pair not yet in Q is added to Q and pushed on A.
//   * Accept states are the reachable pairs in F1 x F2 (§2, Algorithm 1).
//
// Readings where the paper is silent:
//   * Input arcs form a multiset; a listed duplicate joins separately.
//   * Semiring is (+, x) over the reals.  Each product p1*p2 is rounded to
//     float32 (the inputs' precision); merged sums are accumulated in double
//     and rounded to float32 once.
//   * Optional level cap L > 0: only pairs at BFS depth < L are expanded; pairs
//     at depth L are kept as states without outgoing arcs.
//   * Merging never crosses sources (the per-source reduction of Algorithm 2).
//   * Without reduction (§4, the comparison of Table 2 against Table 3): every
//     joined arc pair is its own composed arc with weight fl32(p1 * p2); the
//     reachable states are the same.
//
//   * With epsilon transitions (the paper's §2 excludes them and names
//     composition filters as the way to admit them): one label value eps
//     stands for the empty string on every tape.  Composed states are
//     triples (q1, q2, f) with the filter state f of the three-state epsilon
//     filter of Mohri, Pereira and Riley (also Allauzen, Riley and Schalkwyk
//     2009), which admits exactly one alignment of every pair of paths:
//       - M1 arc with output b != eps and M2 arc with input b: both move,
//         from any f, to f = 0;
//       - M1 arc with output eps and M2 arc with input eps: both move, from
//         f = 0 only, to f = 0;
//       - M1 arc with output eps alone (M2 stays, the composed arc writes
//         eps): from f = 0 or 2, to f = 2;
//       - M2 arc with input eps alone (M1 stays, the composed arc reads
//         eps): from f = 0 or 1, to f = 1.
//     A single move's weight is that arc's weight; accept states are the
//     triples with q1 in F1 and q2 in F2, whatever f.
//
// The merge per source uses an ordered map keyed by (r1, r2, a, c); the pair
// to id map is an ordered map; nothing here is tuned for speed.
//
// Built with: g++ -O2 -std=c++17 -ffp-contract=off -fPIC -shared

#include <algorithm>
#include <array>
#include <chrono>
#include <cstdint>
#include <deque>
#include <map>
#include <utility>
#include <vector>

extern "C" {

struct oracle_fst {
  uint32_t num_states, start, num_isyms, num_osyms;
  uint64_t num_arcs;
  const uint32_t *src, *dst, *ilabel, *olabel;
  const float *weight;
  const uint8_t *final;
};

}  // extern "C"

namespace {

enum { ORACLE_OK = 0, ORACLE_INVALID = 1, ORACLE_ALPHABET = 2 };

struct Result {
  std::vector<std::pair<uint32_t, uint32_t>> pairs;  // id -> (q1, q2)
  std::vector<uint8_t> filt;                          // id -> filter state (epsilon composition)
  std::vector<uint32_t> depth;                        // id -> BFS depth
  std::vector<uint8_t> final;                         // id -> accept
  struct Arc { uint32_t src, dst, a, c; float w; };
  std::vector<Arc> arcs;
  uint64_t premerge = 0;
  uint32_t levels = 0;
  double seconds = 0.0;
};

bool valid(const oracle_fst *m) {
  if (!m || m->num_states == 0 || m->start >= m->num_states) return false;
  if (m->num_arcs && (!m->src || !m->dst || !m->ilabel || !m->olabel || !m->weight))
    return false;
  if (!m->final) return false;
  for (uint64_t e = 0; e < m->num_arcs; ++e) {
    if (m->src[e] >= m->num_states || m->dst[e] >= m->num_states) return false;
    if (m->ilabel[e] >= m->num_isyms || m->olabel[e] >= m->num_osyms) return false;
  }
  return true;
}

// Arc indices of a transducer, grouped for lookup.  by_src: stable order by
// source state.  by_src_in: stable order by (source state, input label).
struct Lookup {
  const oracle_fst *m;
  std::vector<uint32_t> by_src, by_src_in;

  explicit Lookup(const oracle_fst *fst) : m(fst) {
    by_src.resize(m->num_arcs);
    for (uint64_t e = 0; e < m->num_arcs; ++e) by_src[e] = (uint32_t)e;
    by_src_in = by_src;
    std::stable_sort(by_src.begin(), by_src.end(),
                     [&](uint32_t x, uint32_t y) { return m->src[x] < m->src[y]; });
    std::stable_sort(by_src_in.begin(), by_src_in.end(), [&](uint32_t x, uint32_t y) {
      if (m->src[x] != m->src[y]) return m->src[x] < m->src[y];
      return m->ilabel[x] < m->ilabel[y];
    });
  }

  // Arcs leaving q, in input order.
  std::pair<const uint32_t *, const uint32_t *> out(uint32_t q) const {
    auto lo = std::lower_bound(by_src.begin(), by_src.end(), q,
                               [&](uint32_t e, uint32_t v) { return m->src[e] < v; });
    auto hi = std::upper_bound(by_src.begin(), by_src.end(), q,
                               [&](uint32_t v, uint32_t e) { return v < m->src[e]; });
    return {by_src.data() + (lo - by_src.begin()), by_src.data() + (hi - by_src.begin())};
  }

  // Arcs leaving q that read input symbol b, in input order.
  std::pair<const uint32_t *, const uint32_t *> out_reading(uint32_t q, uint32_t b) const {
    auto key_less = [&](uint32_t e, std::pair<uint32_t, uint32_t> v) {
      return std::make_pair(m->src[e], m->ilabel[e]) < v;
    };
    auto less_key = [&](std::pair<uint32_t, uint32_t> v, uint32_t e) {
      return v < std::make_pair(m->src[e], m->ilabel[e]);
    };
    auto lo = std::lower_bound(by_src_in.begin(), by_src_in.end(), std::make_pair(q, b), key_less);
    auto hi = std::upper_bound(by_src_in.begin(), by_src_in.end(), std::make_pair(q, b), less_key);
    return {by_src_in.data() + (lo - by_src_in.begin()),
            by_src_in.data() + (hi - by_src_in.begin())};
  }
};

using ArcKey = std::array<uint32_t, 4>;  // (r1, r2, a, c)

// All composed arcs leaving the pair (q1, q2), merged: the two nested loops of
// Algorithm 1 with the += of its inner statement.  Returns the number of arc
// pairs joined (the unmerged arc count).
uint64_t expand_pair(const Lookup &L1, const Lookup &L2, uint32_t q1, uint32_t q2,
                     std::map<ArcKey, double> &acc) {
  const oracle_fst *m1 = L1.m, *m2 = L2.m;
  uint64_t joined = 0;
  auto r1 = L1.out(q1);
  for (const uint32_t *p = r1.first; p != r1.second; ++p) {
    const uint32_t e1 = *p;
    const uint32_t b = m1->olabel[e1];  // inner symbol written by M1
    auto r2 = L2.out_reading(q2, b);    // M2 arcs reading the same symbol
    for (const uint32_t *s = r2.first; s != r2.second; ++s) {
      const uint32_t e2 = *s;
      const float prod = m1->weight[e1] * m2->weight[e2];
      acc[ArcKey{m1->dst[e1], m2->dst[e2], m1->ilabel[e1], m2->olabel[e2]}] += (double)prod;
      ++joined;
    }
  }
  return joined;
}

// All composed arcs leaving (q1, q2) without reduction: the same two nested
// loops, each joined pair appended as it is found.
struct Joined { uint32_t r1, r2, a, c; float w; };
void expand_pair_unreduced(const Lookup &L1, const Lookup &L2, uint32_t q1, uint32_t q2,
                           std::vector<Joined> &out) {
  const oracle_fst *m1 = L1.m, *m2 = L2.m;
  auto r1 = L1.out(q1);
  for (const uint32_t *p = r1.first; p != r1.second; ++p) {
    const uint32_t e1 = *p;
    auto r2 = L2.out_reading(q2, m1->olabel[e1]);
    for (const uint32_t *s = r2.first; s != r2.second; ++s) {
      const uint32_t e2 = *s;
      out.push_back({m1->dst[e1], m2->dst[e2], m1->ilabel[e1], m2->olabel[e2],
                     m1->weight[e1] * m2->weight[e2]});
    }
  }
}

int compose(const oracle_fst *m1, const oracle_fst *m2, uint32_t max_levels, bool reduce,
            Result &res) {
  if (!valid(m1) || !valid(m2)) return ORACLE_INVALID;
  if (m1->num_osyms != m2->num_isyms) return ORACLE_ALPHABET;
  const auto t0 = std::chrono::steady_clock::now();
  Lookup L1(m1), L2(m2);

  std::map<std::pair<uint32_t, uint32_t>, uint32_t> id;  // the visited set Q
  std::deque<uint32_t> A;                                 // the frontier queue
  const auto s = std::make_pair(m1->start, m2->start);
  id[s] = 0;
  res.pairs.push_back(s);
  res.depth.push_back(0);
  A.push_back(0);

  while (!A.empty()) {
    const uint32_t u = A.front();
    A.pop_front();
    if (max_levels > 0 && res.depth[u] >= max_levels) continue;
    const auto q = res.pairs[u];
    if (!reduce) {
      std::vector<Joined> out;
      expand_pair_unreduced(L1, L2, q.first, q.second, out);
      res.premerge += out.size();
      for (const Joined &j : out) {
        const auto v = std::make_pair(j.r1, j.r2);
        auto it = id.find(v);
        uint32_t vid;
        if (it == id.end()) {
          vid = (uint32_t)res.pairs.size();
          id.emplace(v, vid);
          res.pairs.push_back(v);
          res.depth.push_back(res.depth[u] + 1);
          A.push_back(vid);
        } else {
          vid = it->second;
        }
        res.arcs.push_back({u, vid, j.a, j.c, j.w});
      }
      continue;
    }
    std::map<ArcKey, double> acc;
    res.premerge += expand_pair(L1, L2, q.first, q.second, acc);
    for (const auto &kv : acc) {
      const auto v = std::make_pair(kv.first[0], kv.first[1]);
      auto it = id.find(v);
      uint32_t vid;
      if (it == id.end()) {
        vid = (uint32_t)res.pairs.size();
        id.emplace(v, vid);
        res.pairs.push_back(v);
        res.depth.push_back(res.depth[u] + 1);
        A.push_back(vid);
      } else {
        vid = it->second;
      }
      res.arcs.push_back({u, vid, kv.first[2], kv.first[3], (float)kv.second});
    }
  }
  res.final.resize(res.pairs.size());
  uint32_t maxd = 0;
  for (size_t i = 0; i < res.pairs.size(); ++i) {
    res.final[i] = (m1->final[res.pairs[i].first] && m2->final[res.pairs[i].second]) ? 1 : 0;
    maxd = std::max(maxd, res.depth[i]);
  }
  res.levels = maxd + 1;
  res.seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  return ORACLE_OK;
}

// One composed move out of a triple: target triple, labels, weight.
struct Move { uint32_t r1, r2; uint8_t f; uint32_t a, c; float w; };

// Every move the epsilon filter allows out of (q1, q2, f), in the order M1's
// arcs (with their matches), then M2's input-epsilon arcs alone.
void eps_moves(const Lookup &L1, const Lookup &L2, uint32_t q1, uint32_t q2, uint8_t f,
               uint32_t eps, std::vector<Move> &out) {
  const oracle_fst *m1 = L1.m, *m2 = L2.m;
  auto r1 = L1.out(q1);
  for (const uint32_t *p = r1.first; p != r1.second; ++p) {
    const uint32_t e1 = *p;
    const uint32_t b = m1->olabel[e1];
    if (b != eps || f == 0) {  // both move: on a symbol from any f, on eps from f = 0
      auto r2 = L2.out_reading(q2, b);
      for (const uint32_t *t = r2.first; t != r2.second; ++t) {
        const uint32_t e2 = *t;
        out.push_back({m1->dst[e1], m2->dst[e2], 0, m1->ilabel[e1], m2->olabel[e2],
                       m1->weight[e1] * m2->weight[e2]});
      }
    }
    if (b == eps && (f == 0 || f == 2))  // M1 alone on its output eps
      out.push_back({m1->dst[e1], q2, 2, m1->ilabel[e1], eps, m1->weight[e1]});
  }
  if (f == 0 || f == 1) {  // M2 alone on its input eps
    auto r2 = L2.out_reading(q2, eps);
    for (const uint32_t *t = r2.first; t != r2.second; ++t) {
      const uint32_t e2 = *t;
      out.push_back({q1, m2->dst[e2], 1, eps, m2->olabel[e2], m2->weight[e2]});
    }
  }
}

// Breadth-first search over the triples reachable from (s1, s2, 0); with
// reduce, moves of one source that agree in target triple and labels are
// merged (float64 sum of their float32 weights, rounded once).
int compose_eps(const oracle_fst *m1, const oracle_fst *m2, uint32_t eps, uint32_t max_levels,
                bool reduce, Result &res) {
  if (!valid(m1) || !valid(m2)) return ORACLE_INVALID;
  if (m1->num_osyms != m2->num_isyms) return ORACLE_ALPHABET;
  if (eps >= m1->num_isyms || eps >= m1->num_osyms || eps >= m2->num_osyms) return ORACLE_INVALID;
  const auto t0 = std::chrono::steady_clock::now();
  Lookup L1(m1), L2(m2);
  using Triple = std::array<uint32_t, 3>;
  std::map<Triple, uint32_t> id;
  std::deque<uint32_t> A;
  id[Triple{m1->start, m2->start, 0}] = 0;
  res.pairs.push_back({m1->start, m2->start});
  res.filt.push_back(0);
  res.depth.push_back(0);
  A.push_back(0);
  auto number = [&](uint32_t u, const Move &mv) {
    const Triple v{mv.r1, mv.r2, mv.f};
    auto it = id.find(v);
    if (it != id.end()) return it->second;
    const uint32_t vid = (uint32_t)res.pairs.size();
    id.emplace(v, vid);
    res.pairs.push_back({mv.r1, mv.r2});
    res.filt.push_back(mv.f);
    res.depth.push_back(res.depth[u] + 1);
    A.push_back(vid);
    return vid;
  };
  while (!A.empty()) {
    const uint32_t u = A.front();
    A.pop_front();
    if (max_levels > 0 && res.depth[u] >= max_levels) continue;
    std::vector<Move> moves;
    eps_moves(L1, L2, res.pairs[u].first, res.pairs[u].second, res.filt[u], eps, moves);
    res.premerge += moves.size();
    if (!reduce) {
      for (const Move &mv : moves) res.arcs.push_back({u, number(u, mv), mv.a, mv.c, mv.w});
      continue;
    }
    std::map<std::array<uint32_t, 5>, double> acc;  // (r1, r2, f, a, c)
    for (const Move &mv : moves) acc[{mv.r1, mv.r2, mv.f, mv.a, mv.c}] += (double)mv.w;
    for (const auto &kv : acc) {
      const Move mv{kv.first[0], kv.first[1], (uint8_t)kv.first[2], kv.first[3], kv.first[4], 0.f};
      res.arcs.push_back({u, number(u, mv), mv.a, mv.c, (float)kv.second});
    }
  }
  res.final.resize(res.pairs.size());
  uint32_t maxd = 0;
  for (size_t i = 0; i < res.pairs.size(); ++i) {
    res.final[i] = (m1->final[res.pairs[i].first] && m2->final[res.pairs[i].second]) ? 1 : 0;
    maxd = std::max(maxd, res.depth[i]);
  }
  res.levels = maxd + 1;
  res.seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  return ORACLE_OK;
}

}  // namespace

extern "C" {

// Composition with epsilon transitions: label eps is the empty string on all
// four tapes (it must be a symbol of each alphabet); the composed states are
// (q1, q2, filter state) triples (oracle_filter_states), reachable from
// (start1, start2, 0).  reduce = 0 keeps every move as its own arc.  Returns
// 0, 1 (invalid transducer or eps out of range) or 2 (alphabet mismatch).
int oracle_compose_eps(const oracle_fst *m1, const oracle_fst *m2, uint32_t eps,
                       uint32_t max_levels, int reduce, void **handle) {
  if (!handle) return ORACLE_INVALID;
  *handle = nullptr;
  Result *r = new Result();
  const int rc = compose_eps(m1, m2, eps, max_levels, reduce != 0, *r);
  if (rc != ORACLE_OK) {
    delete r;
    return rc;
  }
  *handle = r;
  return ORACLE_OK;
}

// Per state id: its filter state (0 for results of the other entry points).
void oracle_filter_states(const void *handle, uint8_t *f) {
  const Result *r = static_cast<const Result *>(handle);
  for (size_t i = 0; i < r->pairs.size(); ++i) f[i] = i < r->filt.size() ? r->filt[i] : 0;
}

// Composes m1 with m2 over the pairs reachable from (start1, start2).
// max_levels = 0 means no cap.  On success *handle owns the result (release
// with oracle_free).  Returns 0, 1 (invalid transducer) or 2 (m1's output
// alphabet size differs from m2's input alphabet size).
int oracle_compose(const oracle_fst *m1, const oracle_fst *m2, uint32_t max_levels,
                   void **handle) {
  if (!handle) return ORACLE_INVALID;
  *handle = nullptr;
  Result *r = new Result();
  const int rc = compose(m1, m2, max_levels, true, *r);
  if (rc != ORACLE_OK) {
    delete r;
    return rc;
  }
  *handle = r;
  return ORACLE_OK;
}

// The same search without reduction: every joined arc pair is an arc of the
// result (arcs of a source in join order).
int oracle_compose_unreduced(const oracle_fst *m1, const oracle_fst *m2, uint32_t max_levels,
                             void **handle) {
  if (!handle) return ORACLE_INVALID;
  *handle = nullptr;
  Result *r = new Result();
  const int rc = compose(m1, m2, max_levels, false, *r);
  if (rc != ORACLE_OK) {
    delete r;
    return rc;
  }
  *handle = r;
  return ORACLE_OK;
}

// A batch of source pairs (q1s[i], q2s[i]), i < n, each expanded and merged
// on its own, without any search.  States 0..n-1 of the handle are the
// sources; the distinct targets follow as states n, n+1, ...; arcs carry the
// source's batch index and are ordered by source, then (r1, r2, a, c).
int oracle_expand_pairs(const oracle_fst *m1, const oracle_fst *m2, uint64_t n,
                        const uint32_t *q1s, const uint32_t *q2s, void **handle) {
  if (!handle) return ORACLE_INVALID;
  *handle = nullptr;
  if (!valid(m1) || !valid(m2)) return ORACLE_INVALID;
  if (m1->num_osyms != m2->num_isyms) return ORACLE_ALPHABET;
  for (uint64_t i = 0; i < n; ++i)
    if (q1s[i] >= m1->num_states || q2s[i] >= m2->num_states) return ORACLE_INVALID;
  Result *r = new Result();
  const auto t0 = std::chrono::steady_clock::now();
  Lookup L1(m1), L2(m2);
  for (uint64_t i = 0; i < n; ++i) {
    r->pairs.push_back({q1s[i], q2s[i]});
    r->depth.push_back(0);
  }
  std::map<std::pair<uint32_t, uint32_t>, uint32_t> tid;
  for (uint64_t i = 0; i < n; ++i) {
    std::map<ArcKey, double> acc;
    r->premerge += expand_pair(L1, L2, q1s[i], q2s[i], acc);
    for (const auto &kv : acc) {
      const auto v = std::make_pair(kv.first[0], kv.first[1]);
      auto it = tid.find(v);
      uint32_t vid;
      if (it == tid.end()) {
        vid = (uint32_t)r->pairs.size();
        tid.emplace(v, vid);
        r->pairs.push_back(v);
        r->depth.push_back(1);
      } else {
        vid = it->second;
      }
      r->arcs.push_back({(uint32_t)i, vid, kv.first[2], kv.first[3], (float)kv.second});
    }
  }
  r->final.resize(r->pairs.size());
  for (size_t i = 0; i < r->pairs.size(); ++i)
    r->final[i] = (m1->final[r->pairs[i].first] && m2->final[r->pairs[i].second]) ? 1 : 0;
  r->levels = 2;
  r->seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  *handle = r;
  return ORACLE_OK;
}

// out[0..3] = number of states, arcs (merged unless unreduced), joined arc pairs, BFS layers.
void oracle_counts(const void *handle, uint64_t *out) {
  const Result *r = static_cast<const Result *>(handle);
  out[0] = r->pairs.size();
  out[1] = r->arcs.size();
  out[2] = r->premerge;
  out[3] = r->levels;
}

double oracle_seconds(const void *handle) { return static_cast<const Result *>(handle)->seconds; }

// Per state id: its pair (q1, q2), accept flag and BFS depth.
void oracle_states(const void *handle, uint32_t *q1, uint32_t *q2, uint8_t *final,
                   uint32_t *depth) {
  const Result *r = static_cast<const Result *>(handle);
  for (size_t i = 0; i < r->pairs.size(); ++i) {
    q1[i] = r->pairs[i].first;
    q2[i] = r->pairs[i].second;
    final[i] = r->final[i];
    depth[i] = r->depth[i];
  }
}

// Merged arcs as (source id, target id, input symbol, output symbol, weight).
void oracle_arcs(const void *handle, uint32_t *src, uint32_t *dst, uint32_t *a, uint32_t *c,
                 float *w) {
  const Result *r = static_cast<const Result *>(handle);
  for (size_t i = 0; i < r->arcs.size(); ++i) {
    src[i] = r->arcs[i].src;
    dst[i] = r->arcs[i].dst;
    a[i] = r->arcs[i].a;
    c[i] = r->arcs[i].c;
    w[i] = r->arcs[i].w;
  }
}

void oracle_free(void *handle) { delete static_cast<Result *>(handle); }

}  // extern "C"
