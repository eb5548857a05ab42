"""Fused expand + merge (opts.fused_merge) on the GPU, through the C ABI.

The fused kernel generates each merge tile's composed arcs on chip from the
same match descriptors and CSR arcs, with the same float32 products, and
merges them with the same dense-table merge; tiles the dense table cannot take
are written out and sorted as before.  Sources of the product merge take the
same kernel either way.  So with deterministic ids (within a
depth, ordered by (q1, q2); otherwise the order follows which visited-table
insert wins) a fused composition must equal the unfused one bit for bit (ids,
arc order and weights), and both equal the oracle to the parity bar.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
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


FIELDS = ("q1", "q2", "final", "src", "dst", "a", "c", "w")


def same_bits(x, y, what):
    for f in FIELDS:
        a, b = getattr(x, f), getattr(y, f)
        assert a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8)), \
            f"{what}: field {f} differs between fused and unfused"
    assert x.num_premerge == y.num_premerge


def fused_vs_unfused(F, m1, m2, what, **kw):
    # the fused merge is a per-level kernel: small levels stay off the
    # one-workgroup kernel here so that every level can fuse
    kw.setdefault("small_levels", False)
    fu = F.compose(m1, m2, fused=True, deterministic_ids=True, **kw)
    un = F.compose(m1, m2, fused=False, deterministic_ids=True, **kw)
    same_bits(fu.to_host(), un.to_host(), what)
    return fu


@pytest.mark.parametrize("seed", range(60))
def test_fused_tiny(fstc, seed):
    m1, m2 = tiny_pair(seed)
    g = fused_vs_unfused(fstc, m1, m2, f"tiny {seed}").to_host()
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what=f"tiny {seed}")


@pytest.mark.parametrize("seed", range(40))
def test_fused_config1(fstc, seed):
    m1, m2 = W.config1(seed)
    g = fused_vs_unfused(fstc, m1, m2, f"config1 {seed}").to_host()
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what=f"config1 {seed}")


@pytest.mark.parametrize("cfg,cap", [(4, 3), (2, 3), (3, 0)])
def test_fused_workloads_oracle(fstc, cfg, cap):
    m1, m2 = W.make_config(cfg, 0)
    g = fused_vs_unfused(fstc, m1, m2, f"config{cfg} cap {cap}", max_levels=cap).to_host()
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2, max_levels=cap)),
                what=f"config{cfg} cap {cap}")


@pytest.mark.parametrize("size,target", [("1k", "de"), ("15k", "es")])
def test_fused_paper_pairs(fstc, size, target):
    m1, m2 = W.paper_pair(size, target)
    g = fused_vs_unfused(fstc, m1, m2, f"paper {size} {target}").to_host()
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what=f"paper {size} {target}")


@pytest.mark.timeout(300)
def test_fused_config4_full(fstc):
    """Full HMM-like workload: with the product merge no source has records
    (nothing to fuse); on records every level is fused (one dense tile
    kind); both bit-identical to the unfused composition."""
    m1, m2 = W.config4(0)
    fu = fused_vs_unfused(fstc, m1, m2, "config4 full")
    assert fu.stats["fused_levels"] == 0 and fu.stats["write_launches"] == 0
    assert fu.stats["total_product_records"] == fu.num_premerge_arcs
    fr = fused_vs_unfused(fstc, m1, m2, "config4 full, records only", product=False)
    assert fr.stats["fused_levels"] >= 9 and fr.stats["write_launches"] == 0
    assert fr.stats["total_product_records"] == 0


@pytest.mark.timeout(600)
def test_fused_config2_full(fstc):
    """Medium sparse pair in full: its keys need more bits than the dense
    table takes, so no level is fused and the result is the unfused one."""
    m1, m2 = W.config2(0)
    fu = fused_vs_unfused(fstc, m1, m2, "config2 full")
    assert fu.stats["fused_levels"] == 0


def test_fused_tiles_left_to_sort(fstc):
    """Fused levels whose tiles hold too many sources for the dense table:
    those tiles' arcs are written out and merged by the sort kernel."""
    seen = 0
    for seed in range(200):
        m1, m2 = W.config1(seed)
        fu = fstc.compose(m1, m2, fused=True, small_levels=False)
        if fu.stats["fused_levels"] and fu.stats["total_sort_runs"]:
            fused_vs_unfused(fstc, m1, m2, f"config1 {seed}")
            assert_same(canon_of(fu.to_host()), canon_of(oracle.compose(m1, m2)),
                        what=f"config1 {seed}")
            seen += 1
            if seen == 5:
                break
    assert seen > 0, "no config-1 seed fused a level with sorted tiles"


def test_fused_signed_weights(fstc):
    """Signed, wide-range weights: the exact tile sums match the unfused run."""
    from test_parity_gpu import signed_wide, with_weights
    m1, m2 = W.config4(0)
    rng = np.random.default_rng(78)
    m1 = with_weights(m1, signed_wide(rng, m1.num_arcs, -30, 30))
    m2 = with_weights(m2, signed_wide(rng, m2.num_arcs, -30, 30))
    fused_vs_unfused(fstc, m1, m2, "signed config4 cap 2", max_levels=2)


def with_weights(m, w):
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, m.src, m.dst, m.ilabel,
                 m.olabel, np.asarray(w, np.float32), m.final)


def test_fused_infinite_weights(fstc):
    """Infinite weights on the record path: a fused tile with a non-finite
    product writes its records out for the sort kernel, as the unfused path
    does."""
    m1, m2 = W.config4(0)
    w = m1.weight.copy()
    w[::997] = np.inf
    m1 = with_weights(m1, w)
    fu = fused_vs_unfused(fstc, m1, m2, "config4 inf cap 3", max_levels=3, product=False)
    assert fu.stats["total_sort_runs"] > 0
    g = canon_of(fu.to_host())
    ref = canon_of(oracle.compose(m1, m2, max_levels=3))
    assert_same(g, ref, rtol=np.inf, what="config4 inf cap 3")
    assert np.array_equal(np.isinf(g.w), np.isinf(ref.w))
    fin = np.isfinite(ref.w)
    np.testing.assert_allclose(g.w[fin], ref.w[fin], rtol=1e-5)
