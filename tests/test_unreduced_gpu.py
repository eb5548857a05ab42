"""Composition without reduction on the GPU (opts.no_reduction), through the
C ABI, against the oracle's unreduced composition.

Bar: identical state sets and accept flags, identical arc multisets with
weights bit for bit (each weight is one float32 product on both sides).  At
sizes the oracle cannot finish in seconds, the per-key sums of the unreduced
arcs of sampled sources are compared with the reduced oracle expansion, and
counts and states with the reduced GPU result.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same_multiset, multiset_of
from paper_1805_06383_amd import workloads as W
from test_oracle_pins import tiny_pair

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


def run_unreduced(F, m1, m2, **kw):
    return F.compose(m1, m2, reduce=False, **kw).to_host()


def compare(F, m1, m2, what, **kw):
    g = run_unreduced(F, m1, m2, **kw)
    ref = oracle.compose(m1, m2, reduce=False, **kw)
    assert_same_multiset(multiset_of(g), multiset_of(ref), what=what)
    assert g.num_premerge == ref.num_premerge == g.num_arcs
    if g.num_arcs:
        assert np.all(np.diff(g.src.astype(np.int64)) >= 0), f"{what}: arcs not grouped by source"
    return g


@pytest.mark.parametrize("seed", range(100))
def test_unreduced_tiny(fstc, seed):
    m1, m2 = tiny_pair(seed)
    compare(fstc, m1, m2, f"tiny seed {seed}")


@pytest.mark.parametrize("seed", range(60))
def test_unreduced_config1(fstc, seed):
    m1, m2 = W.config1(seed)
    compare(fstc, m1, m2, f"config1 seed {seed}")


@pytest.mark.parametrize("seed,cap", [(3, 1), (5, 2), (8, 3), (13, 2)])
def test_unreduced_level_cap(fstc, seed, cap):
    m1, m2 = W.config1(seed)
    compare(fstc, m1, m2, f"config1 seed {seed} cap {cap}", max_levels=cap)


@pytest.mark.parametrize("shape", [(3, 4, 5), (1, 1, 1), (16, 64, 16), (40, 300, 7)])
def test_unreduced_matrix_product(fstc, shape):
    """One state: the arcs are all (a, b, c) triples with weight fl32(A[a,b] B[b,c])."""
    rng = np.random.default_rng(sum(shape))
    na, nb, nc = shape
    A = W.random_weights(rng, na * nb).reshape(na, nb)
    B = W.random_weights(rng, nb * nc).reshape(nb, nc)
    g = compare(fstc, W.one_state_dense(A), W.one_state_dense(B), f"matrix {shape}")
    assert g.num_states == 1 and g.num_arcs == na * nb * nc


@pytest.mark.parametrize("cfg,cap", [(4, 2), (4, 3), (2, 2), (3, 0)])
def test_unreduced_workloads(fstc, cfg, cap):
    m1, m2 = W.make_config(cfg, 0)
    compare(fstc, m1, m2, f"config{cfg} cap {cap}", max_levels=cap)


@pytest.mark.parametrize("size,target", [("1k", "de"), ("15k", "it")])
def test_unreduced_paper_pairs(fstc, size, target):
    m1, m2 = W.paper_pair(size, target)
    compare(fstc, m1, m2, f"paper pair {size} {target}")


def test_unreduced_degenerate(fstc):
    rng = np.random.default_rng(4)
    empty1 = W.tiny_random(rng, 3, 2, 2, 0)
    m2 = W.tiny_random(rng, 3, 2, 2, 9)
    g = run_unreduced(fstc, empty1, m2)
    assert g.num_states == 1 and g.num_arcs == 0
    # zero weights are arcs like any other
    m1 = W.tiny_random(rng, 4, 2, 2, 14)
    z = W.FST(m1.num_states, m1.start, m1.num_isyms, m1.num_osyms, m1.src, m1.dst, m1.ilabel,
              m1.olabel, np.zeros_like(m1.weight), m1.final)
    compare(fstc, z, m2, "zero weights")


def test_unreduced_arc_cap(fstc):
    m1, m2 = W.config1(3)
    full = oracle.compose(m1, m2, reduce=False)
    if full.num_arcs > 1:
        with pytest.raises(fstc.FstcError) as e:
            run_unreduced(fstc, m1, m2, max_arcs=full.num_arcs - 1)
        assert e.value.code == fstc.FSTC_ERR_CAPACITY
    compare(fstc, m1, m2, "after the capacity error")


@pytest.mark.timeout(300)
def test_unreduced_config4_full_sampled(fstc):
    """Full-size HMM-like workload without reduction (about 1e9 arcs): states
    equal the reduced run's, every state expands 1024 arc pairs, and for
    sampled sources the unreduced arcs summed per key equal the oracle's
    merged expansion (within 1e-5), with 1024 arcs each."""
    import torch
    m1, m2 = W.config4(0)
    dev = torch.device("cuda:0")
    d1, d2 = fstc.DeviceFST.from_host(m1, dev), fstc.DeviceFST.from_host(m2, dev)
    un = fstc.fstc_compose(d1, d2, reduce=False)
    # the result columns stop at the joined-pair bound (sum over inner symbols
    # of the two inputs' arc counts with that symbol, 1.024e9 arcs of 20 B)
    # instead of growing past it
    h1 = np.bincount(m1.olabel, minlength=m1.num_osyms).astype(np.uint64)
    h2 = np.bincount(m2.ilabel, minlength=m2.num_isyms).astype(np.uint64)
    bound = int((h1 * h2).sum())
    assert un.num_arcs <= bound
    assert un.stats["peak_device_bytes"] < bound * 20 + (2 << 30)
    red = fstc.fstc_compose(d1, d2)
    assert un.num_states == red.num_states
    assert un.num_arcs == un.num_premerge_arcs == red.num_premerge_arcs == 1024 * un.num_states
    pu = torch.stack([un.state_q1, un.state_q2], 1).cpu().numpy().view(np.uint32)
    pr = torch.stack([red.state_q1, red.state_q2], 1).cpu().numpy().view(np.uint32)
    assert np.array_equal(pu[np.lexsort(pu.T[::-1])], pr[np.lexsort(pr.T[::-1])])
    # arcs grouped by source: source id s owns arcs [1024 s, 1024 (s + 1))
    rng = np.random.default_rng(44)
    pick = np.sort(rng.choice(un.num_states, 200, replace=False))
    idx = torch.from_numpy((pick[:, None] * 1024 + np.arange(1024)).ravel()).to(dev)
    src = un.src[idx].cpu().numpy().view(np.uint32)
    assert np.array_equal(src, np.repeat(pick, 1024).astype(np.uint32))
    q1, q2 = pu[:, 0], pu[:, 1]
    dst = un.dst[idx].cpu().numpy().view(np.uint32)
    a = un.ilabel[idx].cpu().numpy().view(np.uint32)
    c = un.olabel[idx].cpu().numpy().view(np.uint32)
    w = un.weight[idx].cpu().numpy()
    rows = np.stack([q1[src], q2[src], q1[dst], q2[dst], a, c], 1).astype(np.int64)
    keys, inv = np.unique(rows, axis=0, return_inverse=True)
    sums = np.zeros(len(keys))
    np.add.at(sums, inv.ravel(), w.astype(np.float64))
    ref = oracle.expand_pairs(m1, m2, q1[pick], q2[pick])
    rk = np.stack([ref.q1[ref.src], ref.q2[ref.src], ref.q1[ref.dst], ref.q2[ref.dst], ref.a,
                   ref.c], 1).astype(np.int64)
    ro = np.lexsort(rk.T[::-1])
    assert np.array_equal(keys, rk[ro])
    np.testing.assert_allclose(sums, ref.w[ro].astype(np.float64), rtol=1e-5)
