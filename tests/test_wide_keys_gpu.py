"""64-bit record keys on the GPU, through the C ABI (§3.4 "Reduction" sorts
packed 64-bit keys).  A composed arc's key is its two part ranks, with as
many bits as the largest part counts of the two inputs need; when they need
more than 32 the records carry u64 keys, which the write pass, the tile sort
merge, the multi-block merge and the composition without reduction each
handle in their own form.  The pair below has start states with 70,000
(target, outer symbol) pairs each (17 + 17 = 34 key bits): the start pair is
a 85,000-record source on the multi-block path, later levels hold small
sources of the hub states on the tile path.  Above 40 bits the library
refuses the inputs with FSTC_ERR_RANGE.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, assert_same_multiset, canon_of, multiset_of
from paper_1805_06383_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


@pytest.fixture(scope="module")
def pair():
    return W.wide_parts_pair(0)


def wide_stats(r):
    assert r.stats["key_bits"] == 34, r.stats["key_bits"]
    assert r.stats["record_key_bytes"] == 8


@pytest.mark.parametrize("cap", [1, 3, 0])
@pytest.mark.parametrize("mode", ["default", "records", "deterministic", "hash"])
def test_wide_keys_reduced(fstc, pair, cap, mode):
    m1, m2 = pair
    kw = {"default": {}, "records": {"product": False},
          "deterministic": {"deterministic_ids": True}, "hash": {"hash_visited": True}}[mode]
    r = fstc.compose(m1, m2, max_levels=cap, **kw)
    wide_stats(r)
    assert r.stats["big_sources"] >= 1  # the start pair's 85,000 records
    g = r.to_host()
    ref = oracle.compose(m1, m2, max_levels=cap)
    assert_same(canon_of(g), canon_of(ref), what=f"wide keys {mode} cap {cap}")
    assert g.num_premerge == ref.num_premerge
    if cap == 1:
        assert ref.num_arcs == 70_000 and ref.num_premerge == 85_000


@pytest.mark.parametrize("cap", [2, 0])
def test_wide_keys_unreduced(fstc, pair, cap):
    m1, m2 = pair
    r = fstc.compose(m1, m2, max_levels=cap, reduce=False)
    wide_stats(r)
    g = r.to_host()
    ref = oracle.compose(m1, m2, max_levels=cap, reduce=False)
    assert_same_multiset(multiset_of(g), multiset_of(ref), what=f"wide keys unreduced cap {cap}")


def test_wide_keys_fused_option(fstc, pair):
    """The fused merge needs short keys; asked for it, levels keep the
    record path and the result is unchanged."""
    m1, m2 = pair
    r = fstc.compose(m1, m2, max_levels=4, fused=True)
    wide_stats(r)
    assert r.stats["fused_levels"] == 0
    assert_same(canon_of(r.to_host()), canon_of(oracle.compose(m1, m2, max_levels=4)),
                what="wide keys fused option")


def test_key_bits_above_40_refused(fstc):
    """Two one-state transducers with 2^20 + 1 parts each need 42 key bits."""
    n = (1 << 20) + 1
    k = np.arange(n)
    z = np.zeros(n)
    w = np.ones(n, np.float32)
    m1 = W.FST(1, 0, n, 4, z, z, k, k % 4, w, [1])
    m2 = W.FST(1, 0, 4, n, z, z, k % 4, k, w, [1])
    with pytest.raises(fstc.FstcError) as e:
        fstc.compose(m1, m2)
    assert e.value.code == fstc.FSTC_ERR_RANGE
    # the library still works afterwards
    a, b = W.config1(1)
    assert fstc.compose(a, b).num_states >= 1
