"""Shape checks of the seeded synthetic workloads (no GPU)."""
import numpy as np
import pytest

from paper_1805_06383_amd import workloads as W


def _check(m):
    assert m.num_arcs == len(m.src)
    if m.num_arcs:
        assert m.src.max() < m.num_states and m.dst.max() < m.num_states
        assert m.ilabel.max() < m.num_isyms and m.olabel.max() < m.num_osyms
        assert m.weight.min() > 0 and m.weight.max() <= 1
    assert m.start < m.num_states


def test_config1_shape_and_determinism():
    m1, m2 = W.config1(7)
    for m in (m1, m2):
        _check(m)
        assert (m.num_states, m.num_arcs) == (200, 2000)
        assert int(m.final.sum()) == 20
    assert (m1.num_isyms, m1.num_osyms, m2.num_isyms, m2.num_osyms) == (50, 100, 100, 50)
    n1, _ = W.config1(7)
    assert n1.digest() == m1.digest()
    assert W.config1(8)[0].digest() != m1.digest()


def test_config2_shape():
    m1, m2 = W.config2(0)
    for m in (m1, m2):
        _check(m)
        assert (m.num_states, m.num_arcs) == (10_000, 200_000)
        assert int(m.final.sum()) == 500
        deg = np.bincount(m.src, minlength=m.num_states)
        assert abs(deg.mean() - 20) < 1e-9 and 3 < deg.std() ** 2 / 20 * 20 < 40
    inner = m1.olabel
    assert m1.num_osyms == 5000 and m2.num_isyms == 5000
    # Zipf(1): symbol 0 is about twice as frequent as symbol 1
    c = np.bincount(inner, minlength=5000)
    assert 1.7 < c[0] / c[1] < 2.3


def test_config3_shape():
    m1, m2 = W.config3(0)
    _check(m1); _check(m2)
    assert m1.num_osyms == 50_000 and m2.num_isyms == 50_000 and m2.num_osyms == 20_000
    assert 330_000 < m1.num_arcs < 420_000
    assert m2.num_states == 1 and 50_000 <= m2.num_arcs <= 250_000
    # one arc per (word, position): the root has one arc per word
    assert int(np.sum(m1.src == 0)) == 50_000
    # word ends accept; every word id is written by exactly len(word) arcs
    assert int(m1.final.sum()) <= 50_000


def test_config4_shape():
    m1, m2 = W.config4(0)
    for m in (m1, m2):
        _check(m)
        assert (m.num_states, m.num_arcs) == (1000, 256_000)
        assert np.all(np.bincount(m.src) == 256)
    # each (state, inner symbol) has exactly 4 arcs
    key = m1.src.astype(np.int64) * 64 + m1.olabel
    assert np.all(np.bincount(key) == 4)
    # (src, dst, in) repeats for every inner symbol: heavy merging downstream
    rows = np.stack([m1.src, m1.dst, m1.ilabel], 1)
    assert len(np.unique(rows, axis=0)) <= 4 * 1000


def test_config5_scaled_shape():
    m1, m2 = W.config5(0, nq=20_000, na=400_000, ng=2_000, nouter=200)
    for m in (m1, m2):
        _check(m)
        assert m.num_arcs == 400_000
        deg = np.bincount(m.src, minlength=m.num_states)
        assert deg.max() > 200  # heavy tail
        assert deg[0] == deg.max()  # the start is a busiest state
        assert int(m.final.sum()) == 200
    p1, p2 = W.config5(0, nq=20_000, na=400_000, ng=2_000, nouter=200, hub_start=False)
    # the relabelling only swaps state 0 with the busiest state
    assert np.array_equal(np.sort(np.bincount(p1.src, minlength=20_000)),
                          np.sort(np.bincount(m1.src, minlength=20_000)))


@pytest.mark.parametrize("size", ["1k", "10k", "15k"])
@pytest.mark.parametrize("target", ["de", "es", "it"])
def test_paper_pair_shape(size, target):
    """Bigram-LM x one-state-TM pairs at the sizes of Table 1."""
    m1, m2 = W.paper_pair(size, target)
    for m in (m1, m2):
        _check(m)
        # an arc's target is the state of its output word (state 0: sentence start)
        assert np.array_equal(m.dst, 1 + m.olabel)
        assert m.num_states == m.num_osyms + 1
    shapes = W.PAPER_SHAPES[size]
    assert (m1.num_states, m1.num_arcs) == shapes["de-en"]
    assert (m2.num_states, m2.num_arcs) == shapes[f"en-{target}"]
    assert m1.num_osyms == m2.num_isyms  # English words join the two
    assert m1.num_isyms == shapes["en-de"][0] - 1  # German source words
    # sparse as in Table 1: arcs are a small fraction of |Q|^2
    assert m1.num_arcs < 0.01 * m1.num_states ** 2
