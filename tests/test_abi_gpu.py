"""The C ABI with the library's own allocator (opts = NULL: stream-ordered
hipMallocAsync / hipFreeAsync) on the GPU: results read back with hipMemcpy
and released with fstc_result_release, against the oracle."""
import ctypes

import numpy as np
import pytest

import oracle
from fstcheck import assert_same, canon_of
from paper_1805_06383_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    hip.hipMemcpy.restype = ctypes.c_int
    hip.hipDeviceSynchronize.restype = ctypes.c_int
    return F, F.load_library(), hip


def read(hip, ptr, n, dtype):
    out = np.empty(n, dtype)
    if n:
        assert hip.hipMemcpy(out.ctypes.data, ptr, out.nbytes, 2) == 0  # device to host
    return out


@pytest.mark.parametrize("case", ["config1", "config4_cap2", "paper_1k"])
def test_default_allocator_round_trip(env, case):
    F, lib, hip = env
    import torch
    if case == "config1":
        m1, m2, cap = *W.config1(3), 0
    elif case == "config4_cap2":
        m1, m2, cap = *W.config4(0), 2
    else:
        m1, m2, cap = *W.paper_pair("1k", "de"), 0
    d1, d2 = F.DeviceFST.from_host(m1, "cuda"), F.DeviceFST.from_host(m2, "cuda")
    torch.cuda.synchronize()
    s1, s2 = d1.struct(), d2.struct()
    opts = F.FstcOpts()
    opts.max_levels = cap
    res = F.FstcResult()
    rc = lib.fstc_compose(ctypes.byref(s1), ctypes.byref(s2), ctypes.byref(opts) if cap else None,
                          None, ctypes.byref(res), None)
    assert rc == 0, lib.fstc_last_error_detail()
    assert hip.hipDeviceSynchronize() == 0
    ns, na = int(res.num_states), int(res.num_arcs)

    class R:
        pass

    g = R()
    g.q1 = read(hip, res.state_q1, ns, np.uint32)
    g.q2 = read(hip, res.state_q2, ns, np.uint32)
    g.final = read(hip, res.final, ns, np.uint8)
    g.src = read(hip, res.src, na, np.uint32)
    g.dst = read(hip, res.dst, na, np.uint32)
    g.a = read(hip, res.ilabel, na, np.uint32)
    g.c = read(hip, res.olabel, na, np.uint32)
    g.w = read(hip, res.weight, na, np.float32)
    g.num_premerge = int(res.num_premerge_arcs)
    lib.fstc_result_release(ctypes.byref(res), ctypes.byref(opts) if cap else None, None)
    assert hip.hipDeviceSynchronize() == 0
    assert not any(res.alloc_ptr) and res.num_arcs == 0  # released and zeroed
    ref = oracle.compose(m1, m2, max_levels=cap)
    assert_same(canon_of(g), canon_of(ref), what=case)
    assert g.num_premerge == ref.num_premerge
    # arcs grouped by source id
    assert np.all(np.diff(g.src.astype(np.int64)) >= 0)


def test_phase_timing(env):
    """Without opts.phase_timing only the single-kernel spans are timed (the
    phase times stay 0); with it every phase is; the result is the same."""
    F, lib, hip = env
    m1, m2 = W.config4(0)
    d1, d2 = F.DeviceFST.from_host(m1, "cuda"), F.DeviceFST.from_host(m2, "cuda")
    a = F.fstc_compose(d1, d2, max_levels=3, small_levels=False)
    b = F.fstc_compose(d1, d2, max_levels=3, phase_timing=True, small_levels=False)
    phases = ("ms_csr", "ms_count", "ms_expand", "ms_merge", "ms_assign")
    assert all(a.stats[k] == 0 for k in phases)
    assert all(b.stats[k] > 0 for k in ("ms_csr", "ms_count", "ms_merge", "ms_assign"))
    for r in (a, b):
        assert r.stats["product_launches"] == 3 and r.stats["ms_product_kernel"] > 0
        assert r.stats["write_launches"] == 0  # every source of config 4 takes the product merge
    assert b.stats["ms_merge"] >= b.stats["ms_product_kernel"]
    x, y = a.to_host(), b.to_host()
    assert x.num_states == y.num_states and len(x.src) == len(y.src)
    assert_same(canon_of(x), canon_of(y), what="phase timing on / off")
