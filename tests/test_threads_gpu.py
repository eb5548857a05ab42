"""Compositions from several host threads at once, each on its own stream,
against the oracle.

A compose call keeps its host-visible staging block, its side streams and its
event pool per calling thread, and its temporaries per call, so calls from
different threads on different streams may overlap on one GPU.  Three threads
run different pairs (a 90-level search that one workgroup runs, a layered
pair whose levels change join classes, and config 4 capped at five levels)
four times each, the calls overlapping, with the record path on one thread;
every result must equal the oracle's composition.
"""
import threading

import pytest

import oracle
from fstcheck import assert_same, canon_of
from paper_1805_06383_amd import workloads as W
from test_join_mix_gpu import join_mix

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fstc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1805_06383_amd import fstc as F
    F.load_library()
    return F


def test_threads_on_their_own_streams(fstc):
    import torch
    m4a, m4b = W.make_config(4)
    jobs = [("config 1 seed 29", W.config1(29), {}),
            ("join mix seed 0", join_mix(0), {"product": False}),
            ("config 4 cap 5", (m4a, m4b), {"max_levels": 5})]
    refs = [oracle.compose(m1, m2, max_levels=kw.get("max_levels", 0))
            for _, (m1, m2), kw in jobs]
    results = [[] for _ in jobs]
    errors = []
    start = threading.Barrier(len(jobs))

    def work(i):
        try:
            name, (m1, m2), kw = jobs[i]
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                d1 = fstc.DeviceFST.from_host(m1, "cuda")
                d2 = fstc.DeviceFST.from_host(m2, "cuda")
                start.wait()
                for _ in range(4):
                    results[i].append(fstc.compose(d1, d2, **kw).to_host())
        except Exception as e:  # reported by the main thread
            errors.append((jobs[i][0], repr(e)))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=100)
    assert not any(t.is_alive() for t in threads), "a compose thread did not finish"
    assert not errors, errors
    for (name, _, _), ref, rs in zip(jobs, refs, results):
        assert len(rs) == 4
        for k, h in enumerate(rs):
            assert_same(canon_of(h), canon_of(ref), rtol=1e-5, what=f"{name} call {k}")
            assert h.num_premerge == ref.num_premerge
