"""Composition with epsilon transitions on the GPU (fstc_compose_eps, through
the C ABI) against the oracle's three-state epsilon filter
(``oracle.compose_eps``): identical triples (q1, q2, filter state), accept
flags and merged arc keys, weights within the parity tolerance; without
merging, identical move multisets bit for bit.  The filter itself is pinned
on the CPU by the weighted relation (tests/test_oracle_eps.py).
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, assert_same_multiset, canon_eps, canon_of, multiset_eps
from paper_1805_06383_amd import workloads as W

pytestmark = pytest.mark.gpu
EPS = 0


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


def check(fstc, m1, m2, what, **kw):
    r = fstc.compose_eps(m1, m2, EPS, **kw)
    g = r.to_host()
    assert g.f is not None and len(g.f) == g.num_states
    ref = oracle.compose_eps(m1, m2, EPS, max_levels=kw.get("max_levels", 0),
                             reduce=kw.get("reduce", True))
    if kw.get("reduce", True):
        assert_same(canon_eps(g), canon_eps(ref), what=what)
    else:
        assert_same_multiset(multiset_eps(g), multiset_eps(ref), what=what)
    assert g.num_premerge == ref.num_premerge, what
    # id 0 is the start triple
    assert (g.q1[0], g.q2[0], g.f[0]) == (m1.start, m2.start, 0)
    return r


def tiny(seed, acyclic):
    rng = np.random.default_rng(9500 + seed)
    nq1, nq2 = (int(x) for x in rng.integers(2, 7, 2))
    p = rng.uniform(0.1, 0.6)
    m1 = W.eps_random(rng, nq1, 3, 4, int(rng.integers(1, 25)), 0.2, p, final_frac=0.5,
                      acyclic=acyclic)
    m2 = W.eps_random(rng, nq2, 4, 3, int(rng.integers(1, 25)), p, 0.2, final_frac=0.5,
                      acyclic=acyclic)
    return m1, m2


@pytest.mark.parametrize("seed", range(60))
def test_tiny_acyclic(fstc, seed):
    m1, m2 = tiny(seed, True)
    check(fstc, m1, m2, f"acyclic {seed}")


@pytest.mark.parametrize("seed", range(60))
def test_tiny_cyclic(fstc, seed):
    m1, m2 = tiny(100 + seed, False)
    check(fstc, m1, m2, f"cyclic {seed}")


@pytest.mark.parametrize("seed", range(12))
def test_config1_shaped(fstc, seed):
    m1, m2 = W.eps_pair(seed)
    check(fstc, m1, m2, f"eps pair {seed}")


@pytest.mark.parametrize("cap", [1, 2, 4])
def test_level_caps(fstc, cap):
    m1, m2 = W.eps_pair(3, eps_inner=0.3)
    check(fstc, m1, m2, f"cap {cap}", max_levels=cap)


@pytest.mark.parametrize("seed", range(6))
def test_without_reduction(fstc, seed):
    m1, m2 = W.eps_pair(seed, nq=60, narcs=400)
    check(fstc, m1, m2, f"unreduced {seed}", reduce=False)


@pytest.mark.parametrize("mode", ["records", "hash", "deterministic"])
def test_modes(fstc, mode):
    m1, m2 = W.eps_pair(5, nq=300, narcs=3000, eps_inner=0.2)
    kw = {"records": {"product": False}, "hash": {"hash_visited": True},
          "deterministic": {"deterministic_ids": True}}[mode]
    check(fstc, m1, m2, f"mode {mode}", **kw)


@pytest.mark.parametrize("cap", [16, 0])
def test_medium_pair(fstc, cap):
    """2,000 states and 40,000 arcs per side, 5% empty inner labels: 303k
    triples at depth 16, 5.4M in the whole search (the oracle takes about a
    minute for it)."""
    m1, m2 = W.eps_pair(11, nq=2000, narcs=40000, nsym=1000, nouter=500, eps_inner=0.05,
                        eps_outer=0.05)
    r = check(fstc, m1, m2, f"medium eps pair, cap {cap}", max_levels=cap)
    assert r.num_states > (300_000 if cap else 5_000_000)


def test_unused_label_is_plain_composition(fstc):
    m1, m2 = W.config1(4)
    for m in (m1, m2):
        m.num_isyms += 1
        m.num_osyms += 1
        m.ilabel = m.ilabel + 1
        m.olabel = m.olabel + 1
    g = fstc.compose_eps(m1, m2, EPS).to_host()
    assert np.all(g.f == 0)
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what="unused empty label")


def test_one_output_eps_meets_one_input_eps(fstc):
    m1 = W.FST(2, 0, 3, 3, [0], [1], [1], [0], [0.5], [0, 1])
    m2 = W.FST(2, 0, 3, 3, [0], [1], [0], [2], [0.25], [0, 1])
    g = fstc.compose_eps(m1, m2, EPS).to_host()
    assert sorted(zip(g.q1.tolist(), g.q2.tolist(), g.f.tolist())) == \
        [(0, 0, 0), (0, 1, 1), (1, 0, 2), (1, 1, 0)]
    arcs = sorted(zip(g.q1[g.dst].tolist(), g.q2[g.dst].tolist(), g.f[g.dst].tolist(),
                      g.a.tolist(), g.c.tolist(), g.w.astype(float).tolist()))
    assert arcs == [(0, 1, 1, 0, 2, 0.25), (1, 0, 2, 1, 0, 0.5), (1, 1, 0, 1, 2, 0.125)]
    assert g.final.tolist() == [int(q1 == 1 and q2 == 1) for q1, q2 in zip(g.q1, g.q2)]


def test_repeat_runs_same(fstc):
    m1, m2 = W.eps_pair(2)
    a = canon_eps(fstc.compose_eps(m1, m2, EPS, deterministic_ids=True).to_host())
    b = canon_eps(fstc.compose_eps(m1, m2, EPS, deterministic_ids=True).to_host())
    assert np.array_equal(a.states, b.states) and np.array_equal(a.keys, b.keys)
    assert np.array_equal(a.w.view(np.uint32), b.w.view(np.uint32))


def test_errors(fstc):
    m1, m2 = W.eps_pair(0)
    with pytest.raises(fstc.FstcError) as e:
        fstc.compose_eps(m1, m2, 50)  # not a symbol of the outer alphabets (50)
    assert e.value.code == fstc.FSTC_ERR_INVALID_ARG
    bad = W.FST(m2.num_states, 0, m2.num_isyms + 1, m2.num_osyms, m2.src, m2.dst, m2.ilabel,
                m2.olabel, m2.weight, m2.final)
    with pytest.raises(fstc.FstcError) as e:
        fstc.compose_eps(m1, bad, EPS)
    assert e.value.code == fstc.FSTC_ERR_ALPHABET
    # the library still works afterwards
    assert fstc.compose_eps(m1, m2, EPS).num_states >= 1
