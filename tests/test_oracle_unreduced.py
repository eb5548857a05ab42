"""Pins for the oracle's composition without reduction (no GPU).

Without reduction (the setting of the paper's Table 2, §4) every joined arc
pair is an arc of the result; reachability is the same as with reduction.
The oracle is checked against:
  * brute force: all-pairs join without merging, trimmed to reachable pairs;
  * one-state transducers: the arcs are exactly the triples (a, b, c) with
    weight fl32(A[a, b] * B[b, c]) (closed form);
  * the reduced oracle: summing the unreduced arcs of each (source, target,
    input, output) key gives the merged weights, and the counts agree.
"""
import numpy as np
import pytest

import oracle
from fstcheck import (assert_same, assert_same_multiset, brute_force_unreduced, canon,
                      canon_of, multiset_of)
from paper_1805_06383_amd import workloads as W
from test_oracle_pins import tiny_pair


@pytest.mark.parametrize("seed", range(200))
def test_unreduced_brute_force_tiny(seed):
    m1, m2 = tiny_pair(seed)
    got = oracle.compose(m1, m2, reduce=False)
    assert_same_multiset(multiset_of(got), multiset_of(brute_force_unreduced(m1, m2)),
                         what=f"seed {seed}")
    assert got.num_arcs == got.num_premerge


@pytest.mark.parametrize("seed", range(30))
@pytest.mark.parametrize("cap", [0, 1, 2])
def test_unreduced_brute_force_config1(seed, cap):
    m1, m2 = W.config1(seed)
    got = oracle.compose(m1, m2, max_levels=cap, reduce=False)
    assert_same_multiset(multiset_of(got), multiset_of(brute_force_unreduced(m1, m2, cap)),
                         what=f"config1 seed {seed} cap {cap}")


@pytest.mark.parametrize("seed", range(6))
def test_unreduced_one_state_closed_form(seed):
    rng = np.random.default_rng(300 + seed)
    na, nb, nc = rng.integers(1, 9, 3)
    A = W.random_weights(rng, na * nb).reshape(na, nb)
    B = W.random_weights(rng, nb * nc).reshape(nb, nc)
    got = oracle.compose(W.one_state_dense(A), W.one_state_dense(B), reduce=False)
    a, b, c = np.meshgrid(np.arange(na), np.arange(nb), np.arange(nc), indexing="ij")
    a, b, c = a.ravel(), b.ravel(), c.ravel()
    w = (A[a, b].astype(np.float32) * B[b, c].astype(np.float32)).astype(np.float32)
    want = np.stack([a, c, w.view(np.uint32).astype(np.int64)], 1)
    have = np.stack([got.a.astype(np.int64), got.c.astype(np.int64),
                     got.w.view(np.uint32).astype(np.int64)], 1)
    assert got.num_states == 1 and np.all(got.src == 0) and np.all(got.dst == 0)
    assert np.array_equal(have[np.lexsort(have.T[::-1])], want[np.lexsort(want.T[::-1])])


@pytest.mark.parametrize("seed", range(60))
def test_unreduced_sums_to_reduced(seed):
    m1, m2 = tiny_pair(1000 + seed) if seed < 40 else W.config1(seed)
    un = oracle.compose(m1, m2, reduce=False)
    red = oracle.compose(m1, m2)
    assert un.num_premerge == red.num_premerge == un.num_arcs
    cu = canon_of(un)
    # sum the unreduced weights of each key in float64
    keys, inv = np.unique(cu.keys, axis=0, return_inverse=True)
    sums = np.zeros(len(keys))
    np.add.at(sums, inv.ravel(), cu.w.astype(np.float64))
    summed = canon(cu.states[:, 0], cu.states[:, 1], cu.finals, *_ids_from_keys(cu, keys), sums)
    assert_same(summed, canon_of(red), rtol=1e-6, what=f"seed {seed}")


def _ids_from_keys(cu, keys):
    """Arc endpoints of canonical keys as ids into the sorted state list."""
    sid = {(int(q1), int(q2)): i for i, (q1, q2) in enumerate(cu.states)}
    src = np.array([sid[(int(k[0]), int(k[1]))] for k in keys], np.int64)
    dst = np.array([sid[(int(k[2]), int(k[3]))] for k in keys], np.int64)
    return src, dst, keys[:, 4], keys[:, 5]
