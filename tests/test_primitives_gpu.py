"""The row-level entry points of the C ABI on the GPU: fstc_exclusive_scan_u64
(the single-pass scan with decoupled look-back the level loop uses) and
fstc_sort_pairs (the stable LSD radix sort of the CSR build), against numpy."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F, torch


# one tile is 2048 elements; 5,000,003 elements are 2,442 tiles, so a tile's
# look-back spans several 64-tile windows
SIZES = [0, 1, 7, 2047, 2048, 2049, 4096 * 3 + 5, 131_072 + 1, 1_000_003, 5_000_003]


@pytest.mark.parametrize("n", SIZES)
def test_exclusive_scan(env, n):
    F, torch = env
    rng = np.random.default_rng(n)
    x = rng.integers(0, 1 << 20, size=n, dtype=np.int64)
    out = F.fstc_exclusive_scan_u64(torch.from_numpy(x).cuda()).cpu().numpy()
    want = np.zeros(n + 1, np.int64)
    np.cumsum(x, out=want[1:])
    assert np.array_equal(out, want)


def test_exclusive_scan_large_values(env):
    """Sums beyond 2^32 and up to 2^60 (64-bit tile totals and prefixes)."""
    F, torch = env
    rng = np.random.default_rng(1)
    x = rng.integers(0, 1 << 40, size=300_001, dtype=np.int64)
    out = F.fstc_exclusive_scan_u64(torch.from_numpy(x).cuda()).cpu().numpy()
    want = np.zeros(len(x) + 1, np.int64)
    np.cumsum(x, out=want[1:])
    assert np.array_equal(out, want)


def test_exclusive_scan_repeated(env):
    """Back-to-back calls reuse freed memory: state words of earlier calls
    must never count as published."""
    F, torch = env
    rng = np.random.default_rng(2)
    for i in range(20):
        n = int(rng.integers(1, 400_000))
        x = rng.integers(0, 1000, size=n, dtype=np.int64)
        out = F.fstc_exclusive_scan_u64(torch.from_numpy(x).cuda()).cpu().numpy()
        assert out[-1] == x.sum() and out[0] == 0
        assert np.array_equal(out[1:], np.cumsum(x)), f"call {i}, n {n}"


@pytest.mark.parametrize("n,lo,hi", [(1, 0, 64), (1000, 0, 64), (4096, 8, 40), (100_003, 0, 64),
                                     (1_000_000, 0, 26), (777, 20, 20)])
def test_sort_pairs(env, n, lo, hi):
    F, torch = env
    rng = np.random.default_rng(n + lo)
    keys = rng.integers(0, 1 << 62, size=n, dtype=np.int64)
    if hi < 64:
        keys &= (1 << hi) - 1  # bits above hi are zero, as the caller promises
    vals = np.arange(n, dtype=np.int32)
    k, v = torch.from_numpy(keys.copy()).cuda(), torch.from_numpy(vals.copy()).cuda()
    F.fstc_sort_pairs(k, v, lo, hi)
    k, v = k.cpu().numpy(), v.cpu().numpy()
    ukeys = keys.view(np.uint64)
    mask = np.uint64((1 << (hi - lo)) - 1) if hi - lo < 64 else np.uint64(~0 & ((1 << 64) - 1))
    field = (ukeys >> np.uint64(lo)) & mask if hi > lo else np.zeros_like(ukeys)
    order = np.argsort(field, kind="stable")
    assert np.array_equal(v, vals[order])
    assert np.array_equal(k, keys[order])
