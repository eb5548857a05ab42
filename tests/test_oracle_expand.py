"""Pins for the oracle's per-source expansion ``oracle.expand_pairs`` (CPU
only).  It is the reference of every sampled comparison at sizes where the
whole search cannot run on the CPU, so it is pinned on its own:

  * brute force over every pair of arcs leaving the two states (§2 arc rule,
    the two inner loops of Algorithm 1), in numpy;
  * the closed form of the HMM-like workload: a source's merged weights are
    the float32 products of its two states' slot-by-symbol weight matrices
    summed over the inner symbol;
  * the batch layout: sources are states 0..n-1 in batch order, distinct
    targets follow from n on, arcs carry the batch index and are grouped by
    it, accept flags follow F1 x F2, the joined count is the sum over the
    batch; repeated sources are expanded again;
  * agreement with the per-source slices of the pinned search (compose).
"""
import numpy as np
import pytest

import oracle
from fstcheck import brute_force_sources, source_rows, weights_close
from paper_1805_06383_amd import workloads as W


def check_batch(res, m1, m2, q1s, q2s, rtol=1e-6):
    """Every property of a correct expansion of the batch (q1s, q2s)."""
    n = len(q1s)
    assert res.num_states >= n
    assert np.array_equal(res.q1[:n], q1s) and np.array_equal(res.q2[:n], q2s), \
        "sources are not states 0..n-1 in batch order"
    tgt = np.stack([res.q1[n:], res.q2[n:]], 1).astype(np.int64)
    if len(tgt):
        assert len(np.unique(tgt, axis=0)) == len(tgt), "a target pair has two ids"
    if res.num_arcs:
        assert np.all(res.src < n), "an arc's source is not a batch index"
        assert np.all(res.dst >= n), "an arc's target is numbered among the sources"
        assert np.all(np.diff(res.src.astype(np.int64)) >= 0), "arcs not grouped by source"
    used = np.zeros(res.num_states, bool)
    used[res.dst] = True
    assert used[n:].all(), "a target state without an arc"
    fin = (m1.final[res.q1] != 0) & (m2.final[res.q2] != 0)
    assert np.array_equal(fin.astype(np.uint8), res.final), "accept flags differ from F1 x F2"
    rows, w, joined = brute_force_sources(m1, m2, q1s, q2s)
    grows, gw = source_rows(res, q1s, q2s)
    assert grows.shape == rows.shape, f"{len(grows)} arcs vs {len(rows)} by brute force"
    assert np.array_equal(grows, rows), "arc keys differ from brute force"
    assert weights_close(gw, w, rtol).all(), "weights differ from brute force"
    assert res.num_premerge == int(joined.sum())


def tiny(seed):
    rng = np.random.default_rng(4000 + seed)
    nq1, nq2 = rng.integers(1, 7, 2)
    m1 = W.tiny_random(rng, int(nq1), 3, 3, int(rng.integers(0, 30)), final_frac=0.5)
    m2 = W.tiny_random(rng, int(nq2), 3, 3, int(rng.integers(0, 30)), final_frac=0.5)
    return m1, m2, rng


@pytest.mark.parametrize("seed", range(60))
def test_tiny_batches(seed):
    m1, m2, rng = tiny(seed)
    k = int(rng.integers(1, 12))
    q1s = rng.integers(0, m1.num_states, k).astype(np.uint32)
    q2s = rng.integers(0, m2.num_states, k).astype(np.uint32)
    check_batch(oracle.expand_pairs(m1, m2, q1s, q2s), m1, m2, q1s, q2s)


def test_repeated_source_is_expanded_again():
    m1, m2 = W.config1(3)
    q1s = np.array([0, 5, 0, 0], np.uint32)
    q2s = np.array([0, 7, 0, 0], np.uint32)
    r = oracle.expand_pairs(m1, m2, q1s, q2s)
    check_batch(r, m1, m2, q1s, q2s)
    per = [np.sum(r.src == i) for i in range(4)]
    assert per[0] == per[2] == per[3]


def test_empty_batch_and_arcless_sources():
    m1, m2 = W.config1(0)
    r = oracle.expand_pairs(m1, m2, np.zeros(0, np.uint32), np.zeros(0, np.uint32))
    assert r.num_states == 0 and r.num_arcs == 0 and r.num_premerge == 0
    empty = W.FST(3, 0, m1.num_osyms, 5, [], [], [], [], [], [1, 0, 1])
    q1s = np.array([0, 1, 2], np.uint32)
    q2s = np.array([0, 1, 2], np.uint32)
    r = oracle.expand_pairs(m1, empty, q1s, q2s)
    assert r.num_states == 3 and r.num_arcs == 0
    check_batch(r, m1, empty, q1s, q2s)


@pytest.mark.parametrize("seed", range(10))
def test_config1_batches(seed):
    m1, m2 = W.config1(seed)
    rng = np.random.default_rng(seed)
    q1s = rng.integers(0, 200, 40).astype(np.uint32)
    q2s = rng.integers(0, 200, 40).astype(np.uint32)
    check_batch(oracle.expand_pairs(m1, m2, q1s, q2s), m1, m2, q1s, q2s)


def config4_closed_form(m1, m2, q1, q2, nsym=64, slots=4):
    """Merged out-arcs of (q1, q2) in the HMM-like workload from its generator
    layout: state q's arcs are laid out by (inner symbol b, slot k), slot k
    carrying one (outer symbol, target) for every b, so the merged weight of
    slots (k, l) is sum over b of fl32(W1[b, k] W2[b, l]); slots of one state
    with the same (outer, target) merge."""
    def state(fst, q, outer_of):
        base = q * nsym * slots
        w = fst.weight[base:base + nsym * slots].reshape(nsym, slots)
        tgt = fst.dst[base:base + slots].astype(np.int64)
        outer = outer_of[base:base + slots].astype(np.int64)
        return w, tgt, outer

    w1, t1, a1 = state(m1, q1, m1.ilabel)
    w2, t2, c2 = state(m2, q2, m2.olabel)
    prod = (w1[:, :, None] * w2[:, None, :]).astype(np.float32).astype(np.float64).sum(0)
    acc = {}
    for k in range(slots):
        for l in range(slots):
            key = (int(t1[k]), int(t2[l]), int(a1[k]), int(c2[l]))
            acc[key] = acc.get(key, 0.0) + prod[k, l]
    keys = sorted(acc)
    return np.array(keys, np.int64), np.array([acc[k] for k in keys], np.float64)


def test_config4_sources_closed_form():
    m1, m2 = W.config4(0)
    rng = np.random.default_rng(44)
    q1s = rng.integers(0, 1000, 25).astype(np.uint32)
    q2s = rng.integers(0, 1000, 25).astype(np.uint32)
    r = oracle.expand_pairs(m1, m2, q1s, q2s)
    check_batch(r, m1, m2, q1s, q2s)
    rows, w = source_rows(r, q1s, q2s)
    for i in range(len(q1s)):
        keys, ref = config4_closed_form(m1, m2, int(q1s[i]), int(q2s[i]))
        sel = rows[:, 0] == i
        assert np.array_equal(rows[sel][:, 3:], keys)
        # two float64 sums of the same float32 products, in two orders
        np.testing.assert_allclose(w[sel].astype(np.float64), ref, rtol=1e-6)
    assert r.num_premerge == 25 * 64 * 4 * 4


@pytest.mark.parametrize("cfg,seed,cap", [(1, 7, 0), (1, 11, 4), (4, 0, 2), (3, 0, 3)])
def test_slices_of_the_search(cfg, seed, cap):
    """The expansion of the search's own expanded states equals the search's
    arcs, source by source (compose is pinned by brute force elsewhere)."""
    m1, m2 = W.make_config(cfg, seed)
    full = oracle.compose(m1, m2, max_levels=cap)
    expanded = np.unique(full.src)
    if len(expanded) > 3000:
        expanded = np.sort(np.random.default_rng(seed).choice(expanded, 3000, replace=False))
    q1s, q2s = full.q1[expanded], full.q2[expanded]
    r = oracle.expand_pairs(m1, m2, q1s, q2s)
    grows, gw = source_rows(r, q1s, q2s)
    pos = np.full(full.num_states, -1, np.int64)
    pos[expanded] = np.arange(len(expanded))
    sel = pos[full.src] >= 0
    src = full.src[sel]; dst = full.dst[sel]
    frows = np.stack([pos[src], full.q1[src], full.q2[src], full.q1[dst], full.q2[dst],
                      full.a[sel], full.c[sel]], 1).astype(np.int64)
    order = np.lexsort(frows.T[::-1])
    assert np.array_equal(grows, frows[order])
    assert np.array_equal(gw, full.w[sel][order])  # same sums in the same order
