"""The one-workgroup small-level kernel (opts.no_small_levels off, the
default) against the per-level kernels and the oracle: levels of at most 512
pairs and 2,048 joined arc pairs are joined, merged, numbered and appended by
one workgroup, several levels per launch, and a level it declines takes the
per-level kernels.  Results must be the same composition either way.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
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


def both(fstc, m1, m2, what, **kw):
    on = fstc.compose(m1, m2, **kw)
    off = fstc.compose(m1, m2, small_levels=False, **kw)
    a, b = on.to_host(), off.to_host()
    assert_same(canon_of(a), canon_of(b), rtol=1e-6, what=f"{what}: small levels on / off")
    assert a.num_premerge == b.num_premerge and a.levels == b.levels
    assert off.stats["small_levels"] == 0
    return on, a


@pytest.mark.parametrize("seed", [0, 3, 7, 29, 30, 41, 77, 132, 150, 199])
def test_config1_seeds(fstc, seed):
    m1, m2 = W.config1(seed)
    on, a = both(fstc, m1, m2, f"config 1 seed {seed}")
    ref = oracle.compose(m1, m2)
    assert_same(canon_of(a), canon_of(ref), what=f"config 1 seed {seed} vs oracle")
    if ref.num_states > 1:
        assert on.stats["small_levels"] == ref.levels - 1 or on.stats["small_levels"] >= 1


def test_whole_search_in_one_launch(fstc):
    """Seed 29: 90 levels of at most a few dozen pairs, all in the kernel."""
    m1, m2 = W.config1(29)
    on, a = both(fstc, m1, m2, "config 1 seed 29")
    assert on.stats["small_levels"] >= 89
    assert on.stats["num_host_syncs"] < 20


@pytest.mark.parametrize("mode", ["deterministic", "hash", "records"])
def test_modes(fstc, mode):
    m1, m2 = W.config1(29)
    kw = {"deterministic": {"deterministic_ids": True}, "hash": {"hash_visited": True},
          "records": {"product": False}}[mode]
    on, a = both(fstc, m1, m2, mode, **kw)
    assert on.stats["small_levels"] > 0
    if mode == "deterministic":
        # ids ordered by (q1, q2) within each depth, as the per-level path numbers them
        off = fstc.compose(m1, m2, small_levels=False, **kw).to_host()
        assert np.array_equal(a.q1, off.q1) and np.array_equal(a.q2, off.q2)


@pytest.mark.parametrize("cap", [1, 2, 5, 20])
def test_level_caps(fstc, cap):
    m1, m2 = W.config1(29)
    on, a = both(fstc, m1, m2, f"cap {cap}", max_levels=cap)
    assert_same(canon_of(a), canon_of(oracle.compose(m1, m2, max_levels=cap)), what=f"cap {cap}")


@pytest.mark.parametrize("size", ["1k", "15k"])
def test_mixed_small_and_large_levels(fstc, size):
    """Paper-shaped pairs: the first level is small, the next ones large, the
    last ones small again."""
    m1, m2 = W.paper_pair(size, "de", 0)
    on, a = both(fstc, m1, m2, f"paper pair {size}")
    assert on.stats["small_levels"] >= 1
    assert_same(canon_of(a), canon_of(oracle.compose(m1, m2)), what=f"paper pair {size}")


@pytest.mark.parametrize("seed", range(40))
def test_tiny_random(fstc, seed):
    rng = np.random.default_rng(8800 + seed)
    m1 = W.tiny_random(rng, int(rng.integers(1, 9)), 3, 3, int(rng.integers(0, 40)), final_frac=0.5)
    m2 = W.tiny_random(rng, int(rng.integers(1, 9)), 3, 3, int(rng.integers(0, 40)), final_frac=0.5)
    on, a = both(fstc, m1, m2, f"tiny {seed}")
    assert_same(canon_of(a), canon_of(oracle.compose(m1, m2)), what=f"tiny {seed}")


def test_state_cap_still_refused(fstc):
    m1, m2 = W.config1(29)
    with pytest.raises(fstc.FstcError) as e:
        fstc.compose(m1, m2, max_states=100)
    assert e.value.code == fstc.FSTC_ERR_CAPACITY
