"""The canonical comparison itself (CPU only): weights that are NaN where the
reference is finite, or infinities of the wrong sign, must fail, so that a
kernel writing garbage can never pass a parity test."""
import numpy as np
import pytest

from fstcheck import assert_same, canon, weights_close


def one_arc(w):
    return canon([0, 1], [0, 0], [0, 1], [0], [1], [0], [0], [np.float32(w)])


GOOD = [(0.5, 0.5), (0.5, 0.5 * (1 + 5e-6)), (np.inf, np.inf), (-np.inf, -np.inf),
        (np.nan, np.nan), (0.0, 0.0), (-0.0, 0.0)]
BAD = [(np.nan, 0.5), (0.25, np.inf), (-np.inf, np.inf), (np.nan, np.inf), (np.inf, 0.5),
       (0.5, np.nan), (np.inf, np.nan), (0.5, 0.5 * (1 + 3e-5)), (1e-30, 0.0)]


@pytest.mark.parametrize("got,ref", GOOD)
def test_close_weights_pass(got, ref):
    assert_same(one_arc(got), one_arc(ref), rtol=1e-5)


@pytest.mark.parametrize("got,ref", BAD)
def test_wrong_weights_fail(got, ref):
    with pytest.raises(AssertionError):
        assert_same(one_arc(got), one_arc(ref), rtol=1e-5)


@pytest.mark.parametrize("got,ref", [(np.nan, 0.5), (np.inf, 0.5), (-np.inf, np.inf),
                                     (0.5, np.nan), (0.5, -np.inf)])
def test_unbounded_tolerance_still_checks_nonfinite(got, ref):
    """rtol = inf skips the size of finite weights, not their pattern."""
    with pytest.raises(AssertionError):
        assert_same(one_arc(got), one_arc(ref), rtol=np.inf)


def test_unbounded_tolerance_accepts_finite():
    assert_same(one_arc(3.0), one_arc(0.0), rtol=np.inf)
    assert_same(one_arc(-7.0), one_arc(1e30), rtol=np.inf)


def test_weights_close_elementwise():
    got = np.array([1.0, np.nan, np.inf, -np.inf, 2.0, 0.0], np.float32)
    ref = np.array([1.0, np.nan, np.inf, np.inf, np.nan, 0.0], np.float32)
    assert weights_close(got, ref, 1e-5).tolist() == [True, True, True, False, False, True]
    assert weights_close(np.float32([2.0**-149]), np.float32([0.0]), 1e-5, atol=2.0**-149).all()
    assert not weights_close(np.float32([2.0**-148]), np.float32([0.0]), 1e-5, atol=2.0**-149).all()
