"""The C-ABI library loads and exports every function include/fstc.h
declares; host-side argument checks return their codes without touching a
GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fstc.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(fstc_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def F():
    from paper_1805_06383_amd import fstc
    if not fstc.LIB_PATH.exists():
        pytest.skip("libfstc.so not built (run __graft_entry__.build())")
    fstc.load_library()
    return fstc


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("fstc_compose", "fstc_result_release", "fstc_build_csr", "fstc_sort_pairs",
              "fstc_exclusive_scan_u64", "fstc_strerror", "fstc_last_error_detail", "fstc_version"):
        assert n in names


def test_every_declared_symbol_is_exported(F):
    lib = ctypes.CDLL(str(F.LIB_PATH))
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(declared_functions()) == set(F.EXPORTS)


def test_version_and_strerror(F):
    assert F.fstc_version() == "0.1.0"
    for code in range(8):
        assert F.fstc_strerror(code)
    assert "unknown" in F.fstc_strerror(99)


def test_struct_layouts_match_header(F):
    # sizes of the structs as the header lays them out (LP64)
    assert ctypes.sizeof(F.FstcFst) == 4 * 4 + 8 + 6 * 8
    assert ctypes.sizeof(F.FstcOpts) == 4 + 4 + 8 + 8 + 3 * 8 + 4 + 4 + 4 + 4 + 4 + 4 + 4 + 4
    assert ctypes.sizeof(F.FstcResult) == 3 * 8 + 4 + 4 + 8 * 8 + 8 * 8 + 8 * 8
    assert ctypes.sizeof(F.FstcStats) == 4 + 4 + 4 * 8 + 8 * 8 + 4 + 4 + 8 + 8 + 4 + 4 + 8 + 4 + 4 + 5 * 8 + 8 + 4 + 4 + 8 + 4 + 4 + 8 + 4 + 4


def test_struct_offsets_match_header(F, tmp_path):
    """Every field of the binding's ctypes structs sits at the offset the C
    header gives it (gcc, LP64), and the structs have the header's sizes."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    structs = {"fstc_fst": F.FstcFst, "fstc_opts": F.FstcOpts, "fstc_result": F.FstcResult,
               "fstc_stats": F.FstcStats}
    lines = ['#include "fstc.h"', "#include <stdio.h>", "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(ROOT, "include")
    r = subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", f"-I{inc}", "-I/opt/rocm/include",
                        str(src), "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, cls in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert got[(cname, fname)] == getattr(cls, fname).offset, (cname, fname)


def _fst(F, **kw):
    base = dict(num_states=4, start=0, num_isyms=3, num_osyms=3, num_arcs=0, src=None, dst=None,
                ilabel=None, olabel=None, weight=None, final=1)
    base.update(kw)
    return F.FstcFst(**base)


def _call(F, m1, m2, opts=None):
    lib = F.load_library()
    out = F.FstcResult()
    rc = lib.fstc_compose(ctypes.byref(m1) if m1 is not None else None,
                          ctypes.byref(m2) if m2 is not None else None,
                          ctypes.byref(opts) if opts is not None else None, None,
                          ctypes.byref(out), None)
    return rc, F.fstc_last_error_detail()


def test_host_validation_codes(F):
    ok = _fst(F)
    assert _call(F, None, ok)[0] == F.FSTC_ERR_INVALID_ARG
    assert _call(F, ok, None)[0] == F.FSTC_ERR_INVALID_ARG
    assert _call(F, _fst(F, num_states=0), ok)[0] == F.FSTC_ERR_INVALID_ARG
    assert _call(F, _fst(F, start=4), ok)[0] == F.FSTC_ERR_INVALID_ARG
    assert _call(F, _fst(F, final=None), ok)[0] == F.FSTC_ERR_INVALID_ARG
    assert _call(F, _fst(F, num_arcs=5), ok)[0] == F.FSTC_ERR_INVALID_ARG  # arrays missing
    rc, msg = _call(F, _fst(F, num_osyms=5), ok)
    assert rc == F.FSTC_ERR_ALPHABET and "num_osyms" in msg
    big = _fst(F, num_arcs=1 << 32, src=1, dst=1, ilabel=1, olabel=1, weight=1)
    assert _call(F, big, ok)[0] == F.FSTC_ERR_RANGE
    # state and symbol ids too wide for the 64-bit CSR keys: 2*32 + 32 bits
    wide = _fst(F, num_states=0xFFFFFFFF, num_isyms=0xFFFFFFFF, num_osyms=3)
    assert _call(F, wide, _fst(F))[0] == F.FSTC_ERR_RANGE
    opts = F.FstcOpts()
    opts.alloc = F.ALLOC_FN(lambda n, c, s: None)  # alloc without free
    assert _call(F, ok, ok, opts)[0] == F.FSTC_ERR_INVALID_ARG
    lib = F.load_library()
    assert lib.fstc_compose(ctypes.byref(ok), ctypes.byref(ok), None, None, None, None) \
        == F.FSTC_ERR_INVALID_ARG


def test_other_entry_points_validate(F):
    lib = F.load_library()
    assert lib.fstc_sort_pairs(None, None, 10, 0, 64, None) == F.FSTC_ERR_INVALID_ARG
    assert lib.fstc_sort_pairs(1, 1, 10, 5, 3, None) == F.FSTC_ERR_INVALID_ARG
    assert lib.fstc_sort_pairs(1, 1, 10, 0, 65, None) == F.FSTC_ERR_INVALID_ARG
    assert lib.fstc_exclusive_scan_u64(None, None, 4, None) == F.FSTC_ERR_INVALID_ARG
    m = _fst(F)
    assert lib.fstc_build_csr(ctypes.byref(m), 1, None, *([None] * 9)) == F.FSTC_ERR_INVALID_ARG


def test_release_of_zeroed_result_is_safe(F):
    r = F.FstcResult()
    F.load_library().fstc_result_release(ctypes.byref(r), None, None)
    assert r.num_states == 0


def test_binding_fails_loudly_without_library(tmp_path):
    from paper_1805_06383_amd import fstc
    with pytest.raises(RuntimeError, match="not built"):
        fstc.load_library(tmp_path / "libfstc.so")
