"""fstc_exclusive_scan_u64_noalloc (the scan entry point that allocates
nothing) against fstc_exclusive_scan_u64, through the C ABI: bit-exact on two
calls in a row, the second with a smaller input (the scratch array keeps the
first call's contents), plus the empty input, a single tile, a ragged
multi-tile size and the size limit."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def F():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc
    fstc.load_library()
    return fstc


def values(n, seed, hi=1 << 40):
    import torch
    rng = np.random.default_rng(seed)
    return torch.from_numpy(rng.integers(0, hi, n, dtype=np.int64)).cuda()


def both(F, x):
    import torch
    ref = F.fstc_exclusive_scan_u64(x)
    out = torch.full((x.numel() + 1,), -1, dtype=torch.int64, device=x.device)
    got = F.fstc_exclusive_scan_u64_noalloc(x, out)
    torch.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy()


def test_two_calls_second_smaller(F):
    for n, seed in ((3_000_001, 1), (100_003, 2)):
        x = values(n, seed)
        got, ref = both(F, x)
        assert np.array_equal(got, ref), f"n = {n}"
        host = np.zeros(n + 1, np.uint64)
        np.cumsum(x.cpu().numpy().astype(np.uint64), out=host[1:])
        assert np.array_equal(got.view(np.uint64), host), f"n = {n}: not the prefix sums"


@pytest.mark.parametrize("n", [0, 1, 2047, 2048, 2049, 65_537])
def test_sizes(F, n):
    got, ref = both(F, values(n, n))
    assert np.array_equal(got, ref)


def test_largest_and_too_large(F):
    import torch
    n = 1 << 28
    x = torch.ones(n, dtype=torch.int64, device="cuda")
    out = torch.empty(n + 1, dtype=torch.int64, device="cuda")
    F.fstc_exclusive_scan_u64_noalloc(x, out)
    assert int(out[n]) == n and int(out[12345]) == 12345
    del x, out
    lib = F.load_library()
    big = (1 << 28) + 1
    rc = lib.fstc_exclusive_scan_u64_noalloc(ctypes.c_void_p(1), ctypes.c_void_p(1), big, None)
    assert rc == F.FSTC_ERR_RANGE
    assert "scratch" in F.fstc_last_error_detail()
    # still usable afterwards
    got, ref = both(F, values(5000, 9))
    assert np.array_equal(got, ref)
