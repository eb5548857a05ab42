"""The two forms of the visited set on the GPU, through the C ABI: the dense
array over all pairs (the default when |Q1| |Q2| <= 2^26) and the hash table
of pair keys (opts.hash_visited, and every larger pair space).  The visited
set only decides which pairs are new and which id a target has, so with
deterministic ids (new pairs numbered by (q1, q2) within each depth) both
give the same composition bit for bit.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, assert_same_multiset, canon_of, multiset_of
from paper_1805_06383_amd import workloads as W
from test_oracle_pins import tiny_pair

pytestmark = pytest.mark.gpu

FIELDS = ("q1", "q2", "final", "src", "dst", "a", "c", "w")


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


def dense_vs_hash(F, m1, m2, what, **kw):
    de = F.compose(m1, m2, deterministic_ids=True, **kw)
    ha = F.compose(m1, m2, deterministic_ids=True, hash_visited=True, **kw)
    pairs = m1.num_states * m2.num_states
    assert de.stats["hash_capacity"] == (pairs if pairs <= 1 << 26 else de.stats["hash_capacity"])
    assert ha.stats["hash_capacity"] & (ha.stats["hash_capacity"] - 1) == 0  # a power of two
    x, y = de.to_host(), ha.to_host()
    for f in FIELDS:
        a, b = getattr(x, f), getattr(y, f)
        assert a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8)), \
            f"{what}: field {f} differs between the dense and the hash visited set"
    assert x.num_premerge == y.num_premerge
    return x


@pytest.mark.parametrize("seed", range(12))
def test_visited_tiny(fstc, seed):
    m1, m2 = tiny_pair(seed)
    g = dense_vs_hash(fstc, m1, m2, f"tiny {seed}")
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what=f"tiny {seed}")


@pytest.mark.parametrize("seed", range(12))
def test_visited_config1(fstc, seed):
    m1, m2 = W.config1(seed)
    g = dense_vs_hash(fstc, m1, m2, f"config1 {seed}")
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2)), what=f"config1 {seed}")


@pytest.mark.parametrize("product", [True, False])
def test_visited_config4(fstc, product):
    m1, m2 = W.config4(0)
    g = dense_vs_hash(fstc, m1, m2, f"config4 cap 3 product={product}", max_levels=3,
                      product=product)
    assert_same(canon_of(g), canon_of(oracle.compose(m1, m2, max_levels=3)),
                what="config4 cap 3")


def test_visited_unreduced(fstc):
    """Without reduction the new pairs come from a claim bitmap over the
    slots: pair indices in the dense form."""
    m1, m2 = W.config4(0)
    g = dense_vs_hash(fstc, m1, m2, "config4 unreduced cap 2", max_levels=2, reduce=False)
    assert_same_multiset(multiset_of(g),
                         multiset_of(oracle.compose(m1, m2, max_levels=2, reduce=False)))


def test_visited_large_pair_space_uses_hash(fstc):
    """A pair space above 2^26 keeps the hash table while the table stays
    smaller than the dense array would be."""
    m1, m2 = W.paper_pair("15k", "de")
    assert m1.num_states * m2.num_states > 1 << 26
    r = fstc.compose(m1, m2)
    cap = r.stats["hash_capacity"]
    assert cap & (cap - 1) == 0 and cap < m1.num_states * m2.num_states
    assert r.stats["visited_form"] == 0


@pytest.mark.parametrize("mode", ["product", "records", "unreduced"])
def test_hash_slots_above_bit30(fstc, mode):
    """A hash table of 2^31 slots (opts.hash_min_log2 = 31, 24 GiB): half of
    its slots have bit 30 set, which no temp entry may read as an id flag
    (the product merge marks known ids that way with the dense array only)."""
    m1, m2 = W.config4(0)
    kw = {"product": {}, "records": {"product": False}, "unreduced": {"reduce": False}}[mode]
    cap = 2 if mode == "unreduced" else 3
    r = fstc.compose(m1, m2, max_levels=cap, hash_visited=True, hash_min_log2=31, **kw)
    assert r.stats["hash_capacity"] == 1 << 31
    assert r.stats["visited_form"] == 0
    if mode == "product":
        assert r.stats["total_product_sources"] > 0
    g = r.to_host()
    if mode == "unreduced":
        ref = oracle.compose(m1, m2, max_levels=cap, reduce=False)
        assert_same_multiset(multiset_of(g), multiset_of(ref), what="2^31 slots unreduced")
    else:
        ref = oracle.compose(m1, m2, max_levels=cap)
        assert_same(canon_of(g), canon_of(ref), what=f"2^31 slots {mode}")
        assert g.num_premerge == ref.num_premerge


def test_hash_min_log2_out_of_range(fstc):
    m1, m2 = W.config1(0)
    with pytest.raises(fstc.FstcError) as e:
        fstc.compose(m1, m2, hash_min_log2=32)
    assert e.value.code == fstc.FSTC_ERR_INVALID_ARG


_HUB = {}


def hub():
    if not _HUB:
        _HUB["m"] = W.hub_pair(0)
    return _HUB["m"]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("cap", [1, 2])
def test_hash_moves_to_dense_array(fstc, cap):
    """A pair space between 2^26 and 2^30 starts with the hash table; the start
    pair's 8.4M composed arcs to 8.4M distinct targets make the grown table
    larger than the dense array over all pairs, so the visited set moves
    there before the level's inserts.  Oracle parity, and with
    deterministic ids the same result bit for bit as with the hash table
    kept throughout."""
    m1, m2 = hub()
    pairs = m1.num_states * m2.num_states
    assert (1 << 26) < pairs <= (1 << 30)
    de = fstc.compose(m1, m2, max_levels=cap, deterministic_ids=True)
    assert de.stats["visited_form"] == 2 and de.stats["hash_capacity"] == pairs
    ha = fstc.compose(m1, m2, max_levels=cap, deterministic_ids=True, hash_visited=True)
    assert ha.stats["visited_form"] == 0
    x, y = de.to_host(), ha.to_host()
    del de, ha
    for f in FIELDS:
        a, b = getattr(x, f), getattr(y, f)
        assert a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8)), \
            f"field {f} differs between the moved and the kept visited set"
    ref = oracle.compose(m1, m2, max_levels=cap)
    assert_same(canon_of(x), canon_of(ref), what=f"hub pair cap {cap}")
    assert x.num_premerge == ref.num_premerge
    r = fstc.compose(m1, m2, max_levels=cap)  # ids in claim order
    assert r.stats["visited_form"] == 2
    assert_same(canon_of(r.to_host()), canon_of(ref), what=f"hub pair cap {cap}, claim order")
