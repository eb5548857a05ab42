"""Pins for the CPU oracle (no GPU): checks against what the paper and the
mathematics fix, independently of how the oracle is written.

  * brute force: all-pairs composition trimmed to reachable pairs (§2, §3.1)
  * one-state transducers: composition is a matrix product (§2 definition)
  * identity transducer: M o Id = accessible part of M with duplicates merged
  * path sums: sum over composed paths x:z = sum_y W1(x, y) W2(y, z)
  * associativity, level-cap monotonicity, degenerate inputs
  * Figure 1 / §3.4 start-pair expansion (golden fixture)
"""
import json
import os

import numpy as np
import pytest

import oracle
from fstcheck import (accessible, assert_same, brute_force, canon, canon_of,
                      label_matrices, path_weights)
from paper_1805_06383_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_pair(seed, nq=(1, 8), ns=(1, 4), ng=(1, 4), nd=(1, 4), na=(0, 30), dups=True):
    rng = np.random.default_rng(seed)
    q1, q2 = rng.integers(*nq, endpoint=True, size=2)
    s, g, d = rng.integers(*ns, endpoint=True), rng.integers(*ng, endpoint=True), \
        rng.integers(*nd, endpoint=True)
    a1, a2 = rng.integers(*na, endpoint=True, size=2)
    m1 = W.tiny_random(rng, int(q1), int(s), int(g), int(a1), final_frac=rng.random())
    m2 = W.tiny_random(rng, int(q2), int(g), int(d), int(a2), final_frac=rng.random())
    if dups and m1.num_arcs > 2:
        # repeat a few arcs verbatim (same src, dst, labels; new weights)
        k = rng.integers(0, m1.num_arcs, 3)
        m1 = W.FST(m1.num_states, m1.start, m1.num_isyms, m1.num_osyms,
                   np.r_[m1.src, m1.src[k]], np.r_[m1.dst, m1.dst[k]],
                   np.r_[m1.ilabel, m1.ilabel[k]], np.r_[m1.olabel, m1.olabel[k]],
                   np.r_[m1.weight, W.random_weights(rng, 3)], m1.final)
    return m1, m2


def as_fst(res, nin, nout, name=""):
    return W.FST(res.num_states, 0, nin, nout, res.src, res.dst, res.a, res.c, res.w,
                 res.final, name=name)


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(300))
def test_brute_force_tiny(seed):
    m1, m2 = tiny_pair(seed)
    ref = brute_force(m1, m2)
    got = oracle.compose(m1, m2)
    assert_same(canon_of(got), canon_of(ref), rtol=1e-6, what=f"seed {seed}")
    # the unmerged count is the number of arc pairs joined from reachable sources
    assert got.num_premerge >= got.num_arcs


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_config1(seed):
    m1, m2 = W.config1(seed)
    ref = brute_force(m1, m2)
    got = oracle.compose(m1, m2)
    assert_same(canon_of(got), canon_of(ref), rtol=1e-6, what=f"config1 seed {seed}")


@pytest.mark.parametrize("seed", range(60))
@pytest.mark.parametrize("cap", [1, 2, 3])
def test_brute_force_level_cap(seed, cap):
    m1, m2 = tiny_pair(1000 + seed, nq=(2, 8), na=(5, 30))
    ref = brute_force(m1, m2, max_levels=cap)
    got = oracle.compose(m1, m2, max_levels=cap)
    assert_same(canon_of(got), canon_of(ref), rtol=1e-6, what=f"seed {seed} cap {cap}")
    assert got.depth.max() <= cap
    assert np.all(got.depth[got.src] < cap)


@pytest.mark.parametrize("seed", range(20))
def test_level_cap_monotone(seed):
    m1, m2 = W.config1(seed)
    full = oracle.compose(m1, m2)
    prev = set()
    for cap in range(1, full.levels + 2):
        r = oracle.compose(m1, m2, max_levels=cap)
        cur = set(zip(r.q1.tolist(), r.q2.tolist()))
        assert prev <= cur
        prev = cur
    assert prev == set(zip(full.q1.tolist(), full.q2.tolist()))
    big = oracle.compose(m1, m2, max_levels=full.levels + 5)
    assert_same(canon_of(big), canon_of(full), rtol=0.0)


@pytest.mark.parametrize("seed", range(10))
def test_matrix_product_closed_form(seed):
    rng = np.random.default_rng(seed)
    na, nb, nc = rng.integers(1, 12, 3)
    W1 = W.random_weights(rng, na * nb).reshape(na, nb)
    W2 = W.random_weights(rng, nb * nc).reshape(nb, nc)
    r = oracle.compose(W.one_state_dense(W1), W.one_state_dense(W2))
    assert r.num_states == 1 and r.final[0] == 1
    assert r.num_arcs == na * nc and r.num_premerge == na * nb * nc
    P = W1.astype(np.float64) @ W2.astype(np.float64)
    np.testing.assert_allclose(r.w.astype(np.float64), P[r.a, r.c], rtol=1e-6)
    assert np.all(r.src == 0) and np.all(r.dst == 0)


@pytest.mark.parametrize("seed", range(30))
@pytest.mark.parametrize("side", ["right", "left"])
def test_identity(seed, side):
    rng = np.random.default_rng(seed)
    m = W.tiny_random(rng, int(rng.integers(1, 10)), 3, 4, int(rng.integers(0, 40)))
    # unique (src, dst, in, out) rows so that x 1.0 keeps weights bit-exact
    rows = np.stack([m.src, m.dst, m.ilabel, m.olabel], 1)
    _, keep = np.unique(rows, axis=0, return_index=True)
    keep = np.sort(keep)
    m = W.FST(m.num_states, m.start, 3, 4, m.src[keep], m.dst[keep], m.ilabel[keep],
              m.olabel[keep], m.weight[keep], m.final)
    acc = accessible(m)
    on = np.isin(m.src, acc)
    if side == "right":
        r = oracle.compose(m, W.identity(m.num_osyms))
        pair = lambda q: (q, 0)  # noqa: E731
        fin_ref = m.final[acc]
    else:
        r = oracle.compose(W.identity(m.num_isyms), m)
        pair = lambda q: (0, q)  # noqa: E731
        fin_ref = m.final[acc]
    q1 = np.array([pair(q)[0] for q in acc]); q2 = np.array([pair(q)[1] for q in acc])
    idx = {q: i for i, q in enumerate(acc)}
    ref = canon(q1, q2, fin_ref, [idx[q] for q in m.src[on]], [idx[q] for q in m.dst[on]],
                m.ilabel[on], m.olabel[on], m.weight[on])
    assert_same(canon_of(r), ref, rtol=0.0, what=f"identity {side} seed {seed}")


@pytest.mark.parametrize("seed", range(12))
def test_identity_merges_duplicates(seed):
    rng = np.random.default_rng(50 + seed)
    m = W.tiny_random(rng, 3, 2, 2, 25)  # many repeated (src, dst, in, out) rows
    r = oracle.compose(m, W.identity(2))
    acc = set(accessible(m))
    sums = {}
    for e in range(m.num_arcs):
        if int(m.src[e]) in acc:
            k = (int(m.src[e]), int(m.dst[e]), int(m.ilabel[e]), int(m.olabel[e]))
            sums[k] = sums.get(k, 0.0) + float(m.weight[e])
    got = {(int(r.q1[s]), int(r.q1[d]), int(a), int(c)): float(w)
           for s, d, a, c, w in zip(r.src, r.dst, r.a, r.c, r.w)}
    assert set(got) == set(sums)
    for k in sums:
        assert abs(got[k] - sums[k]) <= 1e-6 * sums[k]


@pytest.mark.parametrize("seed", range(25))
def test_path_sums(seed):
    rng = np.random.default_rng(700 + seed)
    ns, ng, nd = 2, 2, 2
    m1 = W.tiny_random(rng, int(rng.integers(1, 5)), ns, ng, int(rng.integers(3, 16)))
    m2 = W.tiny_random(rng, int(rng.integers(1, 5)), ng, nd, int(rng.integers(3, 16)))
    r = oracle.compose(m1, m2)
    T1 = label_matrices(m1.num_states, m1.start, ns, ng, m1.src, m1.dst, m1.ilabel,
                        m1.olabel, m1.weight)
    T2 = label_matrices(m2.num_states, m2.start, ng, nd, m2.src, m2.dst, m2.ilabel,
                        m2.olabel, m2.weight)
    Tc = label_matrices(r.num_states, 0, ns, nd, r.src, r.dst, r.a, r.c, r.w)
    for length in range(1, 4):
        for ends in ("any", "final"):
            e1 = np.ones(m1.num_states) if ends == "any" else m1.final.astype(float)
            e2 = np.ones(m2.num_states) if ends == "any" else m2.final.astype(float)
            ec = np.ones(r.num_states) if ends == "any" else r.final.astype(float)
            W1 = path_weights(T1, m1.start, e1, length)   # [x, y]
            W2 = path_weights(T2, m2.start, e2, length)   # [y, z]
            Wc = path_weights(Tc, 0, ec, length)          # [x, z]
            np.testing.assert_allclose(Wc, W1 @ W2, rtol=1e-5, atol=1e-12,
                                       err_msg=f"seed {seed} length {length} {ends}")


@pytest.mark.parametrize("seed", range(15))
def test_associativity(seed):
    rng = np.random.default_rng(900 + seed)
    m1 = W.tiny_random(rng, 4, 2, 3, 14)
    m2 = W.tiny_random(rng, 4, 3, 3, 14)
    m3 = W.tiny_random(rng, 4, 3, 2, 14)
    l12 = oracle.compose(m1, m2)
    left = oracle.compose(as_fst(l12, 2, 3), m3)
    r23 = oracle.compose(m2, m3)
    right = oracle.compose(m1, as_fst(r23, 3, 2))

    def triples(res, inner, nested_left):
        t = []
        for i in range(res.num_states):
            if nested_left:
                j = res.q1[i]
                t.append((inner.q1[j], inner.q2[j], res.q2[i]))
            else:
                j = res.q2[i]
                t.append((res.q1[i], inner.q1[j], inner.q2[j]))
        return t

    tl = triples(left, l12, True)
    tr = triples(right, r23, False)
    sl = {x: i for i, x in enumerate(tl)}
    assert set(tl) == set(tr)
    # relabel right's states to left's ids and compare arcs
    remap = np.array([sl[x] for x in tr])
    kl = {(int(s), int(d), int(a), int(c)): float(w)
          for s, d, a, c, w in zip(left.src, left.dst, left.a, left.c, left.w)}
    kr = {(int(remap[s]), int(remap[d]), int(a), int(c)): float(w)
          for s, d, a, c, w in zip(right.src, right.dst, right.a, right.c, right.w)}
    assert set(kl) == set(kr)
    for k in kl:
        assert abs(kl[k] - kr[k]) <= 1e-5 * kr[k]
    fl = {x: int(left.final[i]) for i, x in enumerate(tl)}
    fr = {x: int(right.final[i]) for i, x in enumerate(tr)}
    assert fl == fr


def test_degenerate_inputs():
    rng = np.random.default_rng(3)
    m1 = W.tiny_random(rng, 3, 2, 2, 6)
    empty = W.FST(2, 1, 2, 2, [], [], [], [], [], [1, 1])
    r = oracle.compose(m1, empty)
    assert r.num_states == 1 and r.num_arcs == 0 and r.num_premerge == 0
    assert (r.q1[0], r.q2[0]) == (m1.start, 1)
    assert r.final[0] == (1 if m1.final[m1.start] else 0)
    r = oracle.compose(empty, W.tiny_random(rng, 2, 2, 2, 5))
    assert r.num_states == 1 and r.num_arcs == 0
    with pytest.raises(oracle.OracleError):
        oracle.compose(m1, W.tiny_random(rng, 2, 3, 2, 5))   # |Gamma| mismatch
    bad = W.FST(2, 0, 2, 2, [0], [5], [0], [0], [0.5], [0, 0])
    with pytest.raises(oracle.OracleError):
        oracle.compose(bad, m1)


def _load_fig1():
    with open(os.path.join(GOLDEN, "figure1.json")) as f:
        g = json.load(f)
    sig = {s: i for i, s in enumerate(g["sigma"])}
    gam = {s: i for i, s in enumerate(g["gamma"])}
    dlt = {s: i for i, s in enumerate(g["delta"])}

    def mk(spec, ins, outs):
        arcs = spec["arcs"]
        fin = np.zeros(spec["num_states"], np.uint8)
        fin[spec["final"]] = 1
        return W.FST(spec["num_states"], spec["start"], len(ins), len(outs),
                     [x[0] for x in arcs], [x[1] for x in arcs], [ins[x[2]] for x in arcs],
                     [outs[x[3]] for x in arcs], [x[4] for x in arcs], fin)

    return g, mk(g["m1"], sig, gam), mk(g["m2"], gam, dlt), sig, gam, dlt


def test_figure1_start_pair():
    g, m1, m2, sig, gam, dlt = _load_fig1()
    r = oracle.compose(m1, m2)
    start = [i for i in range(r.num_arcs) if r.src[i] == 0]
    got = {((int(r.q1[r.dst[i]]), int(r.q2[r.dst[i]])), int(r.a[i]), int(r.c[i])): float(r.w[i])
           for i in start}
    exp = {(tuple(e["dst"]), sig[e["in"]], dlt[e["out"]]): e["weight"]
           for e in g["expected_start_arcs"]}
    assert set(got) == set(exp)
    for k, v in exp.items():
        assert abs(got[k] - v) <= g["weight_tolerance"]
    # no output on gata from the start pair: gata is neither read nor written there
    gata = gam["gata"]
    assert not np.any((m1.src == 0) & (m1.olabel == gata))
    assert not np.any((m2.src == 0) & (m2.ilabel == gata))
    # the figure's unreachable pairs: composing all pairs gives more states
    full = brute_force(m1, m2, max_levels=0)
    assert r.num_states == len(full.q1)
    assert (r.num_states, r.num_arcs) == (4, 4)


def test_figure2_csr_offsets_reading():
    """The CSR fragment of Figure 2, recomputed from the fixture's arcs by a
    plain sort of state 0's arcs on the inner symbol (pins the fixture)."""
    g, m1, m2, sig, gam, dlt = _load_fig1()
    for m, lab, key in ((m1, m1.olabel, "m1_by_output"), (m2, m2.ilabel, "m2_by_input")):
        sel = np.where(m.src == 0)[0]
        inner = np.sort(lab[sel])
        for sym, (off, n) in g["expected_csr_state0"][key].items():
            b = gam[sym]
            assert int(np.searchsorted(inner, b, "left")) == off
            assert int(np.sum(inner == b)) == n
