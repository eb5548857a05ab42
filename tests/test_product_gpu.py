"""Product merge (the default; opts.no_product_merge turns it off) on the GPU,
through the C ABI.

A source whose two states have few (target, outer symbol) parts and whose
arcs fill their (part, inner symbol) cells densely, at most once each, is
merged by one wavefront from its two staged arc matrices: the merged weight
of (p1, p2) is the sum over matched inner symbols g of the float32 products
w1(p1, g) * w2(g, p2) -- exactly the joined arc pairs the record path writes
-- added in float64.  The states, arcs and arc order must equal those of the
record path and of the oracle; weights meet the parity bar (and agree with
the record path to float64 rounding).
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
from paper_1805_06383_amd import workloads as W
from test_oracle_pins import tiny_pair

pytestmark = pytest.mark.gpu

RTOL = 1e-5


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


def with_weights(m, w):
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, m.src, m.dst, m.ilabel,
                 m.olabel, np.asarray(w, np.float32), m.final)


FIELDS = ("q1", "q2", "final", "src", "dst", "a", "c")


def product_vs_records(F, m1, m2, what, rtol=1e-6, **kw):
    """Deterministic ids: identical states, arcs and order with and without
    the product merge; weights within rtol of each other (every level on the
    per-level kernels: the one-workgroup small-level kernel takes neither
    path)."""
    kw.setdefault("small_levels", False)
    pr = F.compose(m1, m2, product=True, deterministic_ids=True, **kw)
    rc = F.compose(m1, m2, product=False, deterministic_ids=True, **kw)
    x, y = pr.to_host(), rc.to_host()
    for f in FIELDS:
        a, b = getattr(x, f), getattr(y, f)
        assert a.shape == b.shape and np.array_equal(a, b), f"{what}: field {f} differs"
    assert x.num_premerge == y.num_premerge, what
    assert rc.stats["total_product_records"] == 0
    np.testing.assert_allclose(x.w, y.w, rtol=rtol, err_msg=what)
    # ids in claim order (levels of product sources alone are then written
    # straight into the result): the same composition, weights bit for bit
    df = F.compose(m1, m2, product=True, **kw)
    a, b = canon_of(df.to_host()), canon_of(x)
    assert np.array_equal(a.states, b.states) and np.array_equal(a.finals, b.finals), what
    assert np.array_equal(a.keys, b.keys), what
    assert np.array_equal(a.w.view(np.uint32), b.w.view(np.uint32)), what
    assert df.num_premerge_arcs == x.num_premerge, what
    return pr


@pytest.mark.parametrize("cap", [1, 2, 3])
def test_product_config4_caps(fstc, cap):
    m1, m2 = W.config4(0)
    pr = product_vs_records(fstc, m1, m2, f"config4 cap {cap}", max_levels=cap)
    st = pr.stats
    assert st["product_launches"] >= 1
    assert st["total_product_records"] == pr.num_premerge_arcs  # every source qualifies
    # 4 parts per state, weights in (0, 1]: every source on the matrix cores
    assert st["total_product_mfma_sources"] == st["total_product_sources"]
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2, max_levels=cap)),
                rtol=RTOL, what=f"config4 cap {cap}")


@pytest.mark.parametrize("seed", range(1, 4))
def test_product_config4_seeds(fstc, seed):
    m1, m2 = W.config4(seed, nq=300)
    pr = product_vs_records(fstc, m1, m2, f"config4 nq 300 seed {seed}")
    assert pr.stats["total_product_sources"] > 0
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2)), rtol=RTOL,
                what=f"config4 nq 300 seed {seed}")


def duplicate_slot(m, every, inner_is_output):
    """Config-4 transducer whose states q % every == 0 carry slot 1 with the
    (outer symbol, target) of slot 0: two arcs in one (part, inner symbol)
    cell, which keeps those states out of the product merge."""
    slots, nq = 4, m.num_states
    per = m.num_arcs // nq  # m * slots arcs per state, slot fastest
    dst, il, ol = m.dst.copy(), m.ilabel.copy(), m.olabel.copy()
    outer = il if inner_is_output else ol
    for q in range(0, nq, every):
        base = q * per + np.arange(0, per, slots)
        dst[base + 1] = dst[base]
        outer[base + 1] = outer[base]
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, m.src, dst, il, ol, m.weight,
                 m.final)


@pytest.mark.parametrize("fused", [False, True])
def test_product_mixed_with_records(fstc, fused):
    """States with parallel arcs in one cell go through records while their
    neighbours take the product merge: both kinds interleave within every
    level (and within merge tiles), and the result is assembled source by
    source."""
    m1, m2 = W.config4(0)
    m1 = duplicate_slot(m1, 3, True)
    m2 = duplicate_slot(m2, 5, False)
    pr = product_vs_records(fstc, m1, m2, "config4 shared cells cap 3", max_levels=3,
                            fused=fused)
    st = pr.stats
    assert 0 < st["total_product_records"] < pr.num_premerge_arcs
    assert st["total_dense_records"] > 0
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2, max_levels=3)),
                rtol=RTOL, what="config4 shared cells cap 3")


def test_product_signed_weights(fstc):
    """Signed weights over a wide range: cancelling float64 sums stay within
    1e-5 of the magnitude sum (the parity bar for signed weights)."""
    from test_parity_gpu import compare_signed, signed_wide
    m1, m2 = W.config4(0)
    rng = np.random.default_rng(79)
    m1 = with_weights(m1, signed_wide(rng, m1.num_arcs, -30, 30))
    m2 = with_weights(m2, signed_wide(rng, m2.num_arcs, -30, 30))
    compare_signed(fstc, m1, m2, "signed config4 cap 2 (product)", max_levels=2)


def test_product_infinite_weights(fstc):
    """Infinite products make infinite sums, as in the oracle's float64 sums."""
    m1, m2 = W.config4(0)
    w = m1.weight.copy()
    w[::997] = np.inf
    m1 = with_weights(m1, w)
    g = fstc.compose(m1, m2, max_levels=3, small_levels=False)
    assert g.stats["total_product_records"] > 0
    gc = canon_of(g.to_host())
    ref = canon_of(oracle.compose(m1, m2, max_levels=3))
    assert_same(gc, ref, rtol=np.inf, what="config4 inf cap 3")
    assert np.array_equal(np.isinf(gc.w), np.isinf(ref.w))
    fin = np.isfinite(ref.w)
    np.testing.assert_allclose(gc.w[fin], ref.w[fin], rtol=RTOL)


def test_product_matrix_product(fstc):
    """One-state transducers: the composition is the matrix product A B; with
    4 + 12 parts on a 40-symbol inner alphabet the single source qualifies."""
    rng = np.random.default_rng(12)
    A = W.random_weights(rng, 4 * 40).reshape(4, 40)
    B = W.random_weights(rng, 40 * 12).reshape(40, 12)
    g = fstc.compose(W.one_state_dense(A), W.one_state_dense(B), small_levels=False)
    assert g.stats["total_product_sources"] == 1
    assert g.stats["total_product_mfma_sources"] == 0  # 12 parts: the vector form
    g = g.to_host()
    assert g.num_premerge == 4 * 40 * 12
    P = A.astype(np.float64) @ B.astype(np.float64)
    np.testing.assert_allclose(g.w.astype(np.float64), P[g.a, g.c], rtol=RTOL)
    assert len(g.w) == 48


@pytest.mark.parametrize("seed", range(30))
def test_product_tiny_and_config1(fstc, seed):
    """Small random pairs (some sources qualify, most do not): same result
    with and without the product merge, equal to the oracle."""
    m1, m2 = tiny_pair(seed) if seed < 15 else W.config1(seed)
    pr = product_vs_records(fstc, m1, m2, f"seed {seed}")
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2)), rtol=RTOL,
                what=f"seed {seed}")


@pytest.mark.parametrize("size,target", [("1k", "de"), ("15k", "it")])
def test_product_paper_pairs(fstc, size, target):
    m1, m2 = W.paper_pair(size, target)
    pr = product_vs_records(fstc, m1, m2, f"paper {size} {target}")
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2)), rtol=RTOL,
                what=f"paper {size} {target}")


@pytest.mark.parametrize("with_inf", [False, True])
def test_product_single_entry(fstc, with_inf):
    """P1 = P2 = 1 on 64 inner symbols: one table entry, all 64 lanes on it
    (one symbol each); with an infinite weight the masked sum runs."""
    rng = np.random.default_rng(21)
    A = W.random_weights(rng, 64).reshape(1, 64)
    B = W.random_weights(rng, 64).reshape(64, 1)
    if with_inf:
        A[0, 17] = np.inf
    g = fstc.compose(W.one_state_dense(A), W.one_state_dense(B), small_levels=False)
    assert g.stats["total_product_sources"] == 1
    # an infinite weight keeps the source off the matrix cores
    assert g.stats["total_product_mfma_sources"] == (0 if with_inf else 1)
    g = g.to_host()
    assert g.num_premerge == 64 and len(g.w) == 1
    ref = oracle.compose(W.one_state_dense(A), W.one_state_dense(B))
    if with_inf:
        assert np.isinf(g.w[0]) and np.isinf(ref.w[0])
    else:
        np.testing.assert_allclose(g.w, ref.w, rtol=RTOL)


def scaled_states(m, every, e):
    """m with the weights of the arcs leaving states q % every == 0 times 2^e."""
    w = m.weight.astype(np.float64).copy()
    w[m.src % every == 0] *= 2.0 ** e
    return with_weights(m, w.astype(np.float32))


@pytest.mark.parametrize("case", ["overflow", "subnormal"])
def test_product_out_of_range_products(fstc, case):
    """Sources whose float32 products would overflow or fall below the
    normal range keep the float32-product (vector) form, where the oracle's
    infinities and subnormal products are reproduced; the others run on the
    matrix cores.  Every weight meets the parity bar (1e-5 relative, plus one
    float32 subnormal step)."""
    m1, m2 = W.config4(0)
    if case == "overflow":
        m1, m2 = scaled_states(m1, 3, 90), scaled_states(m2, 5, 45)
    else:
        m1, m2 = scaled_states(m1, 3, -100), scaled_states(m2, 5, -40)
    g = fstc.compose(m1, m2, max_levels=3, small_levels=False)
    st = g.stats
    assert 0 < st["total_product_mfma_sources"] < st["total_product_sources"]
    gc = canon_of(g.to_host())
    ref = canon_of(oracle.compose(m1, m2, max_levels=3))
    assert_same(gc, ref, rtol=np.inf, what=f"config4 {case} cap 3")
    assert np.array_equal(np.isinf(gc.w), np.isinf(ref.w))
    if case == "overflow":
        assert np.isinf(ref.w).any()
    else:
        assert (np.abs(ref.w) < np.finfo(np.float32).tiny).any()
    fin = np.isfinite(ref.w)
    err = np.abs(gc.w[fin].astype(np.float64) - ref.w[fin].astype(np.float64))
    assert (err <= 1e-5 * np.abs(ref.w[fin].astype(np.float64)) + 2.0 ** -149).all()


def drop_inner(m, every, shift, inner_is_output):
    """m without the arcs of states q % every == 0 whose inner symbol is
    (q + shift) % 64: those states keep one arc per part in each remaining
    segment (still dense) but miss one inner symbol."""
    inner = m.olabel if inner_is_output else m.ilabel
    keep = ~((m.src % every == 0) & (inner == (m.src + shift) % 64))
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, m.src[keep], m.dst[keep],
                 m.ilabel[keep], m.olabel[keep], m.weight[keep], m.final)


def test_product_aligned_lists_differ(fstc):
    """Dense states whose symbol lists have one length but differ (each
    misses another symbol): the aligned form's check fails and the source is
    joined by search; sources whose lists agree take the aligned form.  Same
    result as the record path and the oracle."""
    m1, m2 = W.config4(0)
    m1 = drop_inner(m1, 7, 0, True)
    m2 = drop_inner(m2, 5, 1, False)
    pr = product_vs_records(fstc, m1, m2, "config4 missing symbols cap 4", max_levels=4)
    st = pr.stats
    assert st["total_product_mfma_sources"] == st["total_product_sources"] > 0
    assert_same(canon_of(pr.to_host()), canon_of(oracle.compose(m1, m2, max_levels=4)),
                rtol=RTOL, what="config4 missing symbols cap 4")


def split_halves(m, inner_is_output, flip):
    """m with the arcs of slots 0, 1 kept on inner symbols below 32 and those
    of slots 2, 3 on symbols from 32 on (the reverse when flip): every state
    keeps 4 parts, two arcs per segment."""
    inner = (m.olabel if inner_is_output else m.ilabel).astype(np.int64)
    slot = np.arange(m.num_arcs) % 4
    low = (slot < 2) != flip
    keep = np.where(low, inner < 32, inner >= 32)
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, m.src[keep], m.dst[keep],
                 m.ilabel[keep], m.olabel[keep], m.weight[keep], m.final)


@pytest.mark.parametrize("flip", [False, True])
def test_product_entries_without_terms(fstc, flip):
    """Every source is a product source whose table has entries without a
    term (a part of M1 and a part of M2 sharing no inner symbol): on levels
    of product sources alone the merged arcs are written straight into the
    result, and the entries without a term leave gaps that are closed
    afterwards.  Same result as the record path and the oracle."""
    m1, m2 = W.config4(0, nq=300)
    m1 = split_halves(m1, True, False)
    m2 = split_halves(m2, False, flip)
    pr = product_vs_records(fstc, m1, m2, f"config4 split halves flip={flip}", max_levels=4)
    st = pr.stats
    assert st["total_product_sources"] > 0
    assert st["total_product_records"] == pr.num_premerge_arcs
    g = pr.to_host()
    # the levels of product sources alone were written straight to the result
    assert fstc.compose(m1, m2, max_levels=4, small_levels=False).stats["direct_product_levels"] >= 3
    # fewer merged arcs than table entries: 8 of the 16 entries have terms
    assert g.num_arcs < 16 * len(np.unique(g.src))
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2, max_levels=4)), rtol=RTOL,
                what=f"config4 split halves flip={flip}")


def _with_extra_arc(m, state):
    """m with one more arc at `state`: a copy of its first arc (same inner
    symbol, target and outer symbol, another weight), so that the state's
    (part, symbol) cell holds two arcs and it takes no product merge."""
    j = int(np.flatnonzero(m.src == state)[0])
    def cat(a, v):
        return np.concatenate([np.asarray(a), np.asarray([v], np.asarray(a).dtype)])
    return W.FST(m.num_states, m.start, m.num_isyms, m.num_osyms, cat(m.src, m.src[j]),
                 cat(m.dst, m.dst[j]), cat(m.ilabel, m.ilabel[j]), cat(m.olabel, m.olabel[j]),
                 cat(m.weight, np.float32(0.25)), m.final)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_group_product_levels(fstc, seed):
    """Config-4-shaped pairs: the first levels (at most 64 pairs, all strided
    product sources) are taken whole by one workgroup; the composition equals
    the per-level kernels' and the oracle's."""
    m1, m2 = W.config4(seed, nq=60, m=16, nsym=8, slots=3)
    on = fstc.compose(m1, m2)
    off = fstc.compose(m1, m2, small_levels=False)
    assert on.stats["group_product_levels"] >= 1
    assert off.stats["group_product_levels"] == 0
    a, b = on.to_host(), off.to_host()
    assert_same(canon_of(a), canon_of(b), rtol=1e-6, what=f"seed {seed}: one workgroup / per level")
    assert a.num_premerge == b.num_premerge and a.levels == b.levels
    assert_same(canon_of(a), canon_of(oracle.compose(m1, m2)), rtol=RTOL, what=f"seed {seed} vs oracle")


@pytest.mark.parametrize("depth", [0, 1])
def test_group_product_level_declines(fstc, depth):
    """A pair of another form at depth 0 or 1 (a state with two arcs in one
    cell): the one-workgroup level declines there, the per-level kernels take
    it and the later levels, and the result is unchanged."""
    m1, m2 = W.config4(5, nq=60, m=16, nsym=8, slots=3)
    state = m1.start if depth == 0 else int(m1.dst[np.flatnonzero(m1.src == m1.start)[0]])
    m1 = _with_extra_arc(m1, state)
    on = fstc.compose(m1, m2)
    off = fstc.compose(m1, m2, small_levels=False)
    a, b = on.to_host(), off.to_host()
    assert_same(canon_of(a), canon_of(b), rtol=1e-6, what=f"depth {depth}: declined level")
    assert_same(canon_of(a), canon_of(oracle.compose(m1, m2)), rtol=RTOL, what=f"depth {depth} vs oracle")
    if depth == 0:
        assert on.stats["group_product_levels"] == 0
