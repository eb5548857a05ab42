"""Levels whose join classes change from one level to the next, against the
oracle.

The search of Algorithm 1 joins the inner-symbol lists of the two states of
every pair it expands (Section 4).  The level kernels sort those joins by the
lengths of the two lists into thread, 16-lane group, wave and whole-workgroup
(heavy, more than 2048 symbols on the shorter list) joins, and a level that
follows one without any list join launches its list kernels on a small grid
that loops over the sources.  The workload below is layered so that the
breadth-first levels are, in order: five levels of thread joins only, a level
of about 1,000 pairs mixing heavy, wave, group and thread joins, two levels of
thread joins only, a second mixed level, and a last one.  Both mixed levels
have more heavy joins (about 100 and 75) than the small grid has workgroups
(64), so that grid has to loop.  The second input has
the first one's inner structure (same states, inner symbols and targets, in
another arc order) plus arcs on symbols the first lacks at that state, so that
only pairs (q, q) are reached and every list join has unmatched symbols.
"""
import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
from paper_1805_06383_amd import workloads as W

S = 4096                                    # inner symbols
LAYERS = [1, 4, 16, 64, 256, 1024, 3000, 2000, 2000, 600, 50]
MIXED = (6, 9)                              # layers mixing every join class
HEAVY_MIN = 2048


def join_mix(seed, heavy=300, wide=400, group=800):
    rng = np.random.default_rng(seed)
    base = np.cumsum([0] + LAYERS)
    src, dst, sym = [], [], []
    for k, n in enumerate(LAYERS[:-1]):
        if k in MIXED:
            d = np.full(n, 4)
            i = rng.permutation(n)
            nh = heavy if k == MIXED[0] else heavy // 4
            parts = np.split(i, [nh, nh + wide, nh + wide + group])
            d[parts[0]] = rng.integers(HEAVY_MIN + 1, HEAVY_MIN + 250, len(parts[0]))
            d[parts[1]] = rng.integers(33, 200, len(parts[1]))
            d[parts[2]] = rng.integers(5, 33, len(parts[2]))
        elif k in (7, 8):
            d = rng.integers(1, 3, n)
        else:
            d = np.full(n, 4)
        for j, dj in enumerate(d):
            src.append(np.full(dj, base[k] + j))
            sym.append(rng.choice(S, dj, replace=False))
            dst.append(base[k + 1] + rng.integers(0, LAYERS[k + 1], dj))
    src, dst, sym = np.concatenate(src), np.concatenate(dst), np.concatenate(sym)
    nq, n = int(base[-1]), len(src)
    m1 = W.FST(nq, 0, 16, S, src, dst, rng.integers(0, 16, n), sym,
               rng.uniform(0.1, 1.0, n).astype(np.float32),
               (rng.random(nq) < 0.3).astype(np.uint8))
    p = rng.permutation(n)
    ex, exs = rng.integers(0, nq, n // 8), rng.integers(0, S, n // 8)
    have = set(zip(src.tolist(), sym.tolist()))
    keep = np.array([(a, b) not in have for a, b in zip(ex.tolist(), exs.tolist())], bool)
    ex, exs = ex[keep], exs[keep]
    s2 = np.r_[src[p], ex]
    n2 = len(s2)
    m2 = W.FST(nq, 0, S, 16, s2, np.r_[dst[p], rng.integers(0, nq, len(ex))],
               np.r_[sym[p], exs], rng.integers(0, 16, n2),
               rng.uniform(0.1, 1.0, n2).astype(np.float32),
               (rng.random(nq) < 0.3).astype(np.uint8))
    return m1, m2


def level_classes(m1, ref):
    """Per level of the oracle's search: pairs, and pairs whose list join has
    more than HEAVY_MIN symbols on the shorter (the first input's) list."""
    deg = np.bincount(m1.src, minlength=m1.num_states)
    out = []
    for d in range(int(ref.depth.max()) + 1):
        q = ref.q1[ref.depth == d]
        out.append((len(q), int((deg[q] > HEAVY_MIN).sum())))
    return out


MODES = {"default": {}, "per-level": {"small_levels": False},
         "records": {"product": False}, "deterministic": {"deterministic_ids": True},
         "hash": {"hash_visited": True}}


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


@pytest.fixture(scope="module", params=[0, 5])
def case(request):
    m1, m2 = join_mix(request.param)
    ref = oracle.compose(m1, m2)
    return request.param, m1, m2, ref


def test_workload_shape(case):
    """The levels have the classes the module docstring names."""
    seed, m1, m2, ref = case
    assert np.array_equal(ref.q1, ref.q2)
    lv = level_classes(m1, ref)
    assert len(lv) == len(LAYERS)
    assert all(h == 0 for _, h in lv[:6]) and lv[6][0] > 800
    assert lv[7][1] == 0 and lv[8][1] == 0
    assert lv[6][1] > 64 and lv[9][1] > 64


@pytest.mark.gpu
@pytest.mark.parametrize("mode", list(MODES))
def test_join_classes_change_between_levels(fstc, case, mode):
    seed, m1, m2, ref = case
    g = fstc.compose(m1, m2, **MODES[mode])
    h = g.to_host()
    assert_same(canon_of(h), canon_of(ref), rtol=1e-5, what=f"join mix seed {seed} {mode}")
    assert h.num_premerge == ref.num_premerge
    assert g.stats["num_levels"] >= len(LAYERS) - 1
