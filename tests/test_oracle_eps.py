"""Pins for the oracle's composition with epsilon transitions
(``oracle.compose_eps``, CPU only).

The paper excludes epsilon transitions (§2) and names composition filters as
what admitting them requires; the oracle takes the three-state epsilon filter
(states are triples (q1, q2, f)).  What fixes the result independently of
that construction is the weighted relation: for transducers whose paths are
finite, the composed machine's total weight on every (input string, output
string) pair, with the empty-string label removed from both strings, must be
the sum over middle strings y of M1's weight on (x, y) times M2's on (y, z)
-- every alignment of a pair of paths counted exactly once.  The pins:

  * that relation on random acyclic pairs with the empty-string label on all
    tapes, and on hand-made pairs whose relations are written out;
  * with the label unused, the result is the plain composition (every filter
    state 0, the same arcs bit for bit);
  * without merging, the moves of a source summed per key equal the merged
    arcs; the accept flags are F1 x F2 whatever the filter state.
"""
from collections import defaultdict

import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
from paper_1805_06383_amd import workloads as W

EPS = 0


def relation(n_states, start, final, src, dst, a, c, w, eps=EPS):
    """{(input string, output string): total weight} over the accepting paths
    of an acyclic machine, the empty-string label dropped from both strings
    (weights multiplied and added in float64)."""
    out = defaultdict(list)
    for i in range(len(src)):
        out[int(src[i])].append((int(dst[i]), int(a[i]), int(c[i]), float(w[i])))
    rel = defaultdict(float)
    memo = {}

    def walk(q):
        # {(x, z): weight} of the paths from q to an accept state
        if q in memo:
            return memo[q]
        acc = defaultdict(float)
        if final[q]:
            acc[((), ())] += 1.0
        for (r, ai, ci, wi) in out[q]:
            for (x, z), v in walk(r).items():
                x2 = x if ai == eps else (ai,) + x
                z2 = z if ci == eps else (ci,) + z
                acc[(x2, z2)] += wi * v
        memo[q] = acc
        return acc

    for k, v in walk(start).items():
        rel[k] += v
    return dict(rel)


def fst_relation(m):
    return relation(m.num_states, m.start, m.final, m.src, m.dst, m.ilabel, m.olabel, m.weight)


def result_relation(r):
    return relation(r.num_states, 0, r.final, r.src, r.dst, r.a, r.c, r.w)


def composed_relation(m1, m2):
    r1, r2 = fst_relation(m1), fst_relation(m2)
    by_y = defaultdict(list)
    for (y, z), v in r2.items():
        by_y[y].append((z, v))
    rel = defaultdict(float)
    for (x, y), v in r1.items():
        for z, u in by_y.get(y, ()):
            rel[(x, z)] += v * u
    return dict(rel)


def assert_relations_equal(got, ref, rtol=1e-5):
    keys = set(got) | set(ref)
    for k in keys:
        g, r = got.get(k, 0.0), ref.get(k, 0.0)
        assert abs(g - r) <= rtol * max(abs(r), abs(g)) + 1e-300, \
            f"relation differs at {k}: composed {g!r}, sum over middle strings {r!r}"


def acyclic_pair(seed, eps_in=0.25, eps_inner=0.35, eps_out=0.25):
    rng = np.random.default_rng(9100 + seed)
    nq1, nq2 = (int(x) for x in rng.integers(2, 6, 2))
    m1 = W.eps_random(rng, nq1, 3, 3, int(rng.integers(1, 10)), eps_in, eps_inner,
                      final_frac=0.6, acyclic=True)
    m2 = W.eps_random(rng, nq2, 3, 3, int(rng.integers(1, 10)), eps_inner, eps_out,
                      final_frac=0.6, acyclic=True)
    return m1, m2


@pytest.mark.parametrize("seed", range(150))
def test_relation_random_acyclic(seed):
    m1, m2 = acyclic_pair(seed)
    r = oracle.compose_eps(m1, m2, EPS)
    assert_relations_equal(result_relation(r), composed_relation(m1, m2))


@pytest.mark.parametrize("seed", range(40))
def test_relation_epsilon_heavy(seed):
    """Most inner labels empty: long runs of moves of one side alone and of
    both sides at once, where a filter that admits two orders of the same
    moves, or none, shows."""
    m1, m2 = acyclic_pair(1000 + seed, eps_in=0.3, eps_inner=0.8, eps_out=0.3)
    r = oracle.compose_eps(m1, m2, EPS)
    assert_relations_equal(result_relation(r), composed_relation(m1, m2))


def fst(nq, arcs, finals, nsym=4):
    a = np.array(arcs, dtype=np.float64).reshape(-1, 5) if arcs else np.zeros((0, 5))
    fin = np.zeros(nq, np.uint8)
    fin[list(finals)] = 1
    return W.FST(nq, 0, nsym, nsym, a[:, 0], a[:, 1], a[:, 2], a[:, 3],
                 a[:, 4].astype(np.float32), fin)


def test_one_output_eps_meets_one_input_eps():
    """M1: a:eps/0.5, M2: eps:c/0.25.  Both move at once: one accepting path
    a:c with weight 0.125; the two one-sided moves lead to triples that can
    go no further (the filter forbids the other side's move after them)."""
    m1 = fst(2, [(0, 1, 1, 0, 0.5)], [1])
    m2 = fst(2, [(0, 1, 0, 2, 0.25)], [1])
    r = oracle.compose_eps(m1, m2, EPS)
    assert sorted(zip(r.q1, r.q2, r.f)) == [(0, 0, 0), (0, 1, 1), (1, 0, 2), (1, 1, 0)]
    rel = result_relation(r)
    assert rel == {((1,), (2,)): 0.125}
    arcs = sorted(zip(r.q1[r.dst], r.q2[r.dst], r.f[r.dst], r.a, r.c, r.w.astype(float)))
    assert arcs == [(0, 1, 1, 0, 2, 0.25), (1, 0, 2, 1, 0, 0.5), (1, 1, 0, 1, 2, 0.125)]


def test_two_output_eps_against_one_input_eps():
    """M1 writes nothing on a then b; M2 reads nothing and writes c.  The
    only alignment: both move first (a:c), then M1 alone (b:eps)."""
    m1 = fst(3, [(0, 1, 1, 0, 0.5), (1, 2, 2, 0, 0.75)], [2])
    m2 = fst(2, [(0, 1, 0, 3, 0.25)], [1])
    r = oracle.compose_eps(m1, m2, EPS)
    assert result_relation(r) == {((1, 2), (3,)): 0.5 * 0.75 * 0.25}
    assert composed_relation(m1, m2) == {((1, 2), (3,)): 0.5 * 0.75 * 0.25}


def test_epsilon_then_symbol():
    """M1: a:eps then b:x; M2: x:c.  M1 moves alone, then both on x."""
    m1 = fst(3, [(0, 1, 1, 0, 0.5), (1, 2, 2, 3, 0.5)], [2])
    m2 = fst(2, [(0, 1, 3, 2, 0.5)], [1])
    r = oracle.compose_eps(m1, m2, EPS)
    assert result_relation(r) == {((1, 2), (2,)): 0.125}
    path = sorted(zip(r.q1[r.src], r.q2[r.src], r.f[r.src], r.q1[r.dst], r.q2[r.dst],
                      r.f[r.dst], r.a, r.c))
    assert (0, 0, 0, 1, 0, 2, 1, 0) in path and (1, 0, 2, 2, 1, 0, 2, 2) in path


def test_both_sides_empty_everywhere():
    """M1: eps:eps/0.5 from an accept state to an accept state, M2:
    eps:eps/0.25 likewise.  The relation has the one entry (empty, empty),
    the sum over pairs of paths: both empty (1·1), M1's arc with M2's empty
    path (0.5·1), the reverse (1·0.25) and both arcs (0.5·0.25)."""
    m1 = fst(2, [(0, 1, 0, 0, 0.5)], [0, 1])
    m2 = fst(2, [(0, 1, 0, 0, 0.25)], [0, 1])
    r = oracle.compose_eps(m1, m2, EPS)
    rel = result_relation(r)
    assert set(rel) == {((), ())}
    assert abs(rel[((), ())] - (1 + 0.5 + 0.25 + 0.125)) < 1e-12


@pytest.mark.parametrize("seed", range(30))
def test_unused_label_is_plain_composition(seed):
    m1, m2 = W.config1(seed) if seed < 10 else (None, None)
    if m1 is None:
        rng = np.random.default_rng(seed)
        m1 = W.tiny_random(rng, 5, 4, 4, 25, final_frac=0.5)
        m2 = W.tiny_random(rng, 5, 4, 4, 25, final_frac=0.5)
    # relabel so that no arc carries label 0 on any tape
    for m in (m1, m2):
        m.num_isyms += 1
        m.num_osyms += 1
        m.ilabel = m.ilabel + 1
        m.olabel = m.olabel + 1
    r = oracle.compose_eps(m1, m2, EPS)
    ref = oracle.compose(m1, m2)
    assert np.all(r.f == 0)
    assert r.num_premerge == ref.num_premerge
    assert_same(canon_of(r), canon_of(ref), rtol=0.0, what="unused empty label")


@pytest.mark.parametrize("seed", range(10))
def test_unmerged_moves_sum_to_merged_arcs(seed):
    m1, m2 = W.eps_pair(seed, nq=30, narcs=120, nsym=8, nouter=5, eps_inner=0.3, eps_outer=0.2)
    red = oracle.compose_eps(m1, m2, EPS)
    unr = oracle.compose_eps(m1, m2, EPS, reduce=False)
    assert unr.num_premerge == red.num_premerge == unr.num_arcs
    key = lambda r, i: (int(r.q1[r.src[i]]), int(r.q2[r.src[i]]), int(r.f[r.src[i]]),
                        int(r.q1[r.dst[i]]), int(r.q2[r.dst[i]]), int(r.f[r.dst[i]]),
                        int(r.a[i]), int(r.c[i]))
    sums = defaultdict(float)
    for i in range(unr.num_arcs):
        sums[key(unr, i)] += float(unr.w[i])
    assert len(sums) == red.num_arcs
    for i in range(red.num_arcs):
        assert abs(np.float32(sums[key(red, i)]) - red.w[i]) <= 1e-6 * abs(red.w[i])
    fin = m1.final[red.q1] & m2.final[red.q2]
    assert np.array_equal(fin, red.final)
    assert set(np.unique(red.f)) <= {0, 1, 2}


def test_level_cap_and_errors():
    m1, m2 = W.eps_pair(3, nq=40, narcs=160, nsym=8, nouter=5)
    full = oracle.compose_eps(m1, m2, EPS)
    capped = oracle.compose_eps(m1, m2, EPS, max_levels=2)
    assert capped.num_states <= full.num_states
    assert capped.depth.max() <= 2
    with pytest.raises(oracle.OracleError):
        oracle.compose_eps(m1, m2, 5)  # 5 is not a symbol of the outer alphabets
