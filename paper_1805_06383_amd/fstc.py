"""Python binding of libfstc.so (declared in include/fstc.h).

Argument marshalling only: every step of the composition runs in the HIP
library.  PyTorch provides device memory (its caching allocator, through the
allocator callbacks of ``fstc_opts``) and the stream.  Unsigned 32-bit arrays
are carried in ``torch.int32`` tensors holding the same bits.

Names follow the C ABI: ``fstc_compose``, ``fstc_result_release``,
``fstc_build_csr``, ``fstc_sort_pairs``, ``fstc_exclusive_scan_u64``,
``fstc_exclusive_scan_u64_noalloc``,
``fstc_strerror``, ``fstc_last_error_detail``, ``fstc_version``; ``compose``
is the convenience entry point.
"""
from __future__ import annotations

import ctypes
import threading
from dataclasses import dataclass, field
from pathlib import Path

import numpy as np
import torch

LIB_PATH = Path(__file__).resolve().with_name("libfstc.so")

FSTC_OK = 0
FSTC_ERR_INVALID_ARG = 1
FSTC_ERR_ALPHABET = 2
FSTC_ERR_RANGE = 3
FSTC_ERR_CAPACITY = 4
FSTC_ERR_OOM = 5
FSTC_ERR_HIP = 6
FSTC_ERR_INTERNAL = 7


class FstcError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[fstc error {code}] {msg}")
        self.code = code


_vp = ctypes.c_void_p
_u32, _u64 = ctypes.c_uint32, ctypes.c_uint64
ALLOC_FN = ctypes.CFUNCTYPE(_vp, ctypes.c_size_t, _vp, _vp)
FREE_FN = ctypes.CFUNCTYPE(None, _vp, ctypes.c_size_t, _vp, _vp)


class FstcFst(ctypes.Structure):
    _fields_ = [("num_states", _u32), ("start", _u32), ("num_isyms", _u32), ("num_osyms", _u32),
                ("num_arcs", _u64), ("src", _vp), ("dst", _vp), ("ilabel", _vp),
                ("olabel", _vp), ("weight", _vp), ("final", _vp)]


class FstcOpts(ctypes.Structure):
    _fields_ = [("max_levels", _u32), ("deterministic_ids", _u32), ("max_states", _u64),
                ("max_arcs", _u64), ("alloc", ALLOC_FN), ("free", FREE_FN), ("alloc_ctx", _vp),
                ("no_reduction", _u32), ("fused_merge", _u32), ("no_product_merge", _u32),
                ("hash_visited", _u32), ("phase_timing", _u32), ("hash_min_log2", _u32),
                ("no_small_levels", _u32)]


class FstcResult(ctypes.Structure):
    _fields_ = [("num_states", _u64), ("num_arcs", _u64), ("num_premerge_arcs", _u64),
                ("num_levels", _u32), ("reserved0", _u32),
                ("state_q1", _vp), ("state_q2", _vp), ("final", _vp), ("src", _vp),
                ("dst", _vp), ("ilabel", _vp), ("olabel", _vp), ("weight", _vp),
                ("alloc_ptr", _vp * 8), ("alloc_bytes", ctypes.c_size_t * 8)]


class FstcStats(ctypes.Structure):
    _fields_ = [("num_levels", _u32), ("num_host_syncs", _u32), ("max_frontier", _u64),
                ("max_level_premerge", _u64), ("big_sources", _u64), ("hash_capacity", _u64),
                ("ms_total", ctypes.c_double), ("ms_csr", ctypes.c_double),
                ("ms_count", ctypes.c_double), ("ms_expand", ctypes.c_double),
                ("ms_merge", ctypes.c_double), ("ms_assign", ctypes.c_double),
                ("ms_write_kernel", ctypes.c_double), ("ms_merge_kernel", ctypes.c_double),
                ("write_launches", _u32), ("merge_launches", _u32),
                ("total_matches", _u64), ("total_big_records", _u64),
                ("record_key_bytes", _u32), ("key_bits", _u32),
                ("ms_sort_kernel", ctypes.c_double), ("sort_launches", _u32), ("fused_levels", _u32),
                ("total_dense_records", _u64), ("total_dense_runs", _u64),
                ("total_sort_runs", _u64), ("total_product_records", _u64),
                ("total_product_sources", _u64), ("ms_product_kernel", ctypes.c_double),
                ("product_launches", _u32), ("visited_form", _u32),
                ("total_product_mfma_sources", _u64), ("direct_product_levels", _u32),
                ("small_levels", _u32), ("peak_device_bytes", _u64),
                ("group_product_levels", _u32), ("reserved2", _u32)]


EXPORTS = ("fstc_compose", "fstc_compose_eps", "fstc_result_release", "fstc_build_csr", "fstc_sort_pairs",
           "fstc_exclusive_scan_u64", "fstc_exclusive_scan_u64_noalloc", "fstc_strerror",
           "fstc_last_error_detail", "fstc_version")

_lib = None


def load_library(path: Path | str | None = None) -> ctypes.CDLL:
    """Loads libfstc.so; raises if it has not been built (no fallback)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = Path(path) if path else LIB_PATH
    if not p.exists():
        raise RuntimeError(f"{p} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(str(p))
    lib.fstc_compose.argtypes = [ctypes.POINTER(FstcFst), ctypes.POINTER(FstcFst),
                                 ctypes.POINTER(FstcOpts), _vp, ctypes.POINTER(FstcResult),
                                 ctypes.POINTER(FstcStats)]
    lib.fstc_compose.restype = ctypes.c_int
    lib.fstc_compose_eps.argtypes = [ctypes.POINTER(FstcFst), ctypes.POINTER(FstcFst), _u32,
                                     ctypes.POINTER(FstcOpts), _vp, ctypes.POINTER(FstcResult),
                                     ctypes.POINTER(_vp), ctypes.POINTER(FstcStats)]
    lib.fstc_compose_eps.restype = ctypes.c_int
    lib.fstc_result_release.argtypes = [ctypes.POINTER(FstcResult), ctypes.POINTER(FstcOpts), _vp]
    lib.fstc_result_release.restype = None
    lib.fstc_build_csr.argtypes = [ctypes.POINTER(FstcFst), ctypes.c_int, _vp] + [_vp] * 9
    lib.fstc_build_csr.restype = ctypes.c_int
    lib.fstc_sort_pairs.argtypes = [_vp, _vp, _u64, ctypes.c_int, ctypes.c_int, _vp]
    lib.fstc_sort_pairs.restype = ctypes.c_int
    lib.fstc_exclusive_scan_u64.argtypes = [_vp, _vp, _u64, _vp]
    lib.fstc_exclusive_scan_u64.restype = ctypes.c_int
    lib.fstc_exclusive_scan_u64_noalloc.argtypes = [_vp, _vp, _u64, _vp]
    lib.fstc_exclusive_scan_u64_noalloc.restype = ctypes.c_int
    lib.fstc_strerror.argtypes = [ctypes.c_int]
    lib.fstc_strerror.restype = ctypes.c_char_p
    lib.fstc_last_error_detail.argtypes = []
    lib.fstc_last_error_detail.restype = ctypes.c_char_p
    lib.fstc_version.argtypes = []
    lib.fstc_version.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def fstc_strerror(code: int) -> str:
    return load_library().fstc_strerror(code).decode()


def fstc_last_error_detail() -> str:
    return load_library().fstc_last_error_detail().decode()


def fstc_version() -> str:
    return load_library().fstc_version().decode()


def _check(rc: int):
    if rc != FSTC_OK:
        raise FstcError(rc, f"{fstc_strerror(rc)}: {fstc_last_error_detail()}")


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


# ---------------------------------------------------------------------------
class TorchAllocator:
    """fstc_opts allocator callbacks backed by PyTorch's caching allocator.

    Each allocation is a uint8 tensor on the device and the stream of the
    call; it stays alive in ``live`` until the library frees it.  Buffers the
    library hands back in a result are taken out of ``live`` by the caller.
    """

    def __init__(self, device: torch.device):
        self.device = device
        self.live: dict[int, torch.Tensor] = {}
        self._alloc = ALLOC_FN(self._do_alloc)
        self._free = FREE_FN(self._do_free)

    def _do_alloc(self, nbytes, ctx, stream):
        try:
            t = torch.empty(int(nbytes), dtype=torch.uint8, device=self.device)
        except RuntimeError:
            return None
        p = t.data_ptr()
        self.live[p] = t
        return p

    def _do_free(self, ptr, nbytes, ctx, stream):
        self.live.pop(int(ptr), None)

    def take(self, ptr) -> torch.Tensor | None:
        if not ptr:
            return None
        return self.live.pop(int(ptr))

    def opts(self, max_levels=0, deterministic_ids=False, max_states=0, max_arcs=0,
             reduce=True, fused=False, product=True, hash_visited=False,
             phase_timing=False, hash_min_log2=0, small_levels=True) -> FstcOpts:
        return FstcOpts(int(max_levels), 1 if deterministic_ids else 0, int(max_states),
                        int(max_arcs), self._alloc, self._free, None, 0 if reduce else 1,
                        1 if fused else 0, 0 if product else 1, 1 if hash_visited else 0,
                        1 if phase_timing else 0, int(hash_min_log2),
                        0 if small_levels else 1)


_ALLOCATORS: dict = {}


def _allocator(device: torch.device) -> TorchAllocator:
    """One TorchAllocator per thread and device, reused by every call (making the two
    ctypes callbacks costs tens of microseconds).  Between calls it holds no
    allocation: a call's temporaries are freed by the library and its result
    buffers taken out by _wrap."""
    key = (threading.get_ident(), device.type,
           device.index if device.index is not None else torch.cuda.current_device())
    a = _ALLOCATORS.get(key)
    if a is None:
        a = _ALLOCATORS[key] = TorchAllocator(device)
    a.live.clear()  # a call that failed may have left entries behind
    return a


# ---------------------------------------------------------------------------
@dataclass
class DeviceFST:
    """A transducer whose arc arrays live on the GPU (see workloads.FST)."""

    num_states: int
    start: int
    num_isyms: int
    num_osyms: int
    src: torch.Tensor
    dst: torch.Tensor
    ilabel: torch.Tensor
    olabel: torch.Tensor
    weight: torch.Tensor
    final: torch.Tensor

    @property
    def num_arcs(self) -> int:
        return int(self.src.numel())

    @classmethod
    def from_host(cls, m, device="cuda") -> "DeviceFST":
        def u32(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.uint32).view(np.int32)).to(device)
        return cls(int(m.num_states), int(m.start), int(m.num_isyms), int(m.num_osyms),
                   u32(m.src), u32(m.dst), u32(m.ilabel), u32(m.olabel),
                   torch.from_numpy(np.ascontiguousarray(m.weight, np.float32)).to(device),
                   torch.from_numpy(np.ascontiguousarray(m.final, np.uint8)).to(device))

    def struct(self) -> FstcFst:
        def ptr(t):
            return t.data_ptr() if t.numel() else None
        return FstcFst(self.num_states, self.start, self.num_isyms, self.num_osyms,
                       self.num_arcs, ptr(self.src), ptr(self.dst), ptr(self.ilabel),
                       ptr(self.olabel), ptr(self.weight), self.final.data_ptr())


@dataclass
class Composed:
    """Result of fstc_compose as device tensors (int32 tensors hold u32 bits)."""

    num_states: int
    num_arcs: int
    num_premerge_arcs: int
    num_levels: int
    state_q1: torch.Tensor
    state_q2: torch.Tensor
    final: torch.Tensor
    src: torch.Tensor
    dst: torch.Tensor
    ilabel: torch.Tensor
    olabel: torch.Tensor
    weight: torch.Tensor
    stats: dict = field(default_factory=dict)
    state_filter: torch.Tensor | None = None  # uint8 filter state (fstc_compose_eps)

    def to_host(self):
        """numpy view: q1, q2, final, src, dst, a, c, w (uint32 / float32),
        and f (filter states) for a composition with epsilon transitions."""
        def u(t):
            return t.cpu().numpy().view(np.uint32)
        return HostComposed(u(self.state_q1), u(self.state_q2), self.final.cpu().numpy(),
                            u(self.src), u(self.dst), u(self.ilabel), u(self.olabel),
                            self.weight.cpu().numpy(), self.num_premerge_arcs, self.num_levels,
                            None if self.state_filter is None
                            else self.state_filter.cpu().numpy())


@dataclass
class HostComposed:
    q1: np.ndarray
    q2: np.ndarray
    final: np.ndarray
    src: np.ndarray
    dst: np.ndarray
    a: np.ndarray
    c: np.ndarray
    w: np.ndarray
    num_premerge: int
    levels: int
    f: np.ndarray | None = None

    @property
    def num_states(self):
        return len(self.q1)

    @property
    def num_arcs(self):
        return len(self.src)


_ESIZE = {torch.int32: 4, torch.float32: 4, torch.uint8: 1}


def _view(buf: torch.Tensor | None, n: int, dtype, device) -> torch.Tensor:
    if buf is None or n == 0:
        return torch.empty(0, dtype=dtype, device=device)
    return buf[: n * _ESIZE[dtype]].view(dtype)


def fstc_compose(m1: DeviceFST, m2: DeviceFST, max_levels: int = 0,
                 deterministic_ids: bool = False, max_states: int = 0, max_arcs: int = 0,
                 stream=None, want_stats: bool = True, reduce: bool = True,
                 fused: bool = False, product: bool = True,
                 hash_visited: bool = False, phase_timing: bool = False,
                 hash_min_log2: int = 0, small_levels: bool = True) -> Composed:
    """Reachable composition m1 o m2 on the GPU (see fstc_compose in fstc.h).
    reduce=False keeps every joined arc pair as its own arc (opts.no_reduction);
    fused=True merges tiles without writing their composed arcs first
    (opts.fused_merge); product=False sends every source through written
    records (opts.no_product_merge); hash_visited=True keeps the visited set
    in the hash table even for small pair spaces (opts.hash_visited);
    phase_timing=True fills the per-phase times of the stats
    (opts.phase_timing; the kernel times are always there); hash_min_log2 > 0
    gives the hash table at least 2^hash_min_log2 slots (opts.hash_min_log2);
    small_levels=False sends every level through the per-level kernels
    (opts.no_small_levels)."""
    lib = load_library()
    device = m1.src.device if m1.num_arcs else m1.final.device
    alloc = _allocator(device)
    opts = alloc.opts(max_levels, deterministic_ids, max_states, max_arcs, reduce, fused, product,
                      hash_visited, phase_timing, hash_min_log2, small_levels)
    s1, s2 = m1.struct(), m2.struct()
    res = FstcResult()
    st = FstcStats()
    rc = lib.fstc_compose(ctypes.byref(s1), ctypes.byref(s2), ctypes.byref(opts),
                          _stream_handle(stream), ctypes.byref(res),
                          ctypes.byref(st) if want_stats else None)
    _check(rc)
    return _wrap(res, st if want_stats else None, alloc, device)


def fstc_compose_eps(m1: DeviceFST, m2: DeviceFST, eps: int, max_levels: int = 0,
                     deterministic_ids: bool = False, max_states: int = 0, max_arcs: int = 0,
                     stream=None, want_stats: bool = True, reduce: bool = True,
                     fused: bool = False, product: bool = True,
                     hash_visited: bool = False) -> Composed:
    """Composition with epsilon transitions (see fstc_compose_eps in fstc.h):
    label ``eps`` is the empty string on every tape; states are triples, the
    filter state in ``state_filter``.  Options as for fstc_compose."""
    lib = load_library()
    device = m1.src.device if m1.num_arcs else m1.final.device
    alloc = _allocator(device)
    opts = alloc.opts(max_levels, deterministic_ids, max_states, max_arcs, reduce, fused, product,
                      hash_visited, False, 0)
    s1, s2 = m1.struct(), m2.struct()
    res = FstcResult()
    st = FstcStats()
    filt = _vp()
    rc = lib.fstc_compose_eps(ctypes.byref(s1), ctypes.byref(s2), int(eps), ctypes.byref(opts),
                              _stream_handle(stream), ctypes.byref(res), ctypes.byref(filt),
                              ctypes.byref(st) if want_stats else None)
    _check(rc)
    return _wrap(res, st if want_stats else None, alloc, device, filt.value)


def _wrap(res, st, alloc, device, filt_ptr=None) -> Composed:
    """A result of the C ABI as tensors that own its allocations."""
    ns, na = int(res.num_states), int(res.num_arcs)
    owners = [(int(res.alloc_ptr[i]), alloc.take(res.alloc_ptr[i])) for i in range(8)
              if res.alloc_ptr[i]]
    assert not alloc.live, f"library left {len(alloc.live)} temporaries allocated"
    i32, f32, u8 = torch.int32, torch.float32, torch.uint8

    typed = {}  # (allocation, dtype) -> the allocation viewed as dtype

    def view(ptr, n, dtype):
        """Tensor of n elements at device address ptr, inside the allocation
        that owns it (the result arrays may share allocations): a slice of
        that allocation viewed as dtype (one view per allocation and dtype;
        allocations are whole multiples of 256 bytes)."""
        if not ptr or n == 0:
            return torch.empty(0, dtype=dtype, device=device)
        ptr = int(ptr)
        es = _ESIZE[dtype]
        for k, (base, buf) in enumerate(owners):
            if base <= ptr < base + buf.numel():
                off = ptr - base
                if off % es or buf.numel() % es:
                    return _view(buf[off:], n, dtype, device)
                t = typed.get((k, dtype))
                if t is None:
                    t = typed[(k, dtype)] = buf.view(dtype)
                return t[off // es: off // es + n]
        raise RuntimeError("result array outside its recorded allocations")

    stats = {k: getattr(st, k) for k, _ in FstcStats._fields_} if st is not None else {}
    return Composed(ns, na, int(res.num_premerge_arcs), int(res.num_levels),
                    view(res.state_q1, ns, i32), view(res.state_q2, ns, i32),
                    view(res.final, ns, u8), view(res.src, na, i32), view(res.dst, na, i32),
                    view(res.ilabel, na, i32), view(res.olabel, na, i32),
                    view(res.weight, na, f32), stats,
                    view(filt_ptr, ns, u8) if filt_ptr is not None else None)


def fstc_result_release(result: FstcResult, opts: FstcOpts | None = None, stream=None):
    """Frees a raw FstcResult obtained through the C ABI (not needed for
    Composed, whose tensors own their memory)."""
    load_library().fstc_result_release(ctypes.byref(result),
                                       ctypes.byref(opts) if opts is not None else None,
                                       _stream_handle(stream))


def compose(m1, m2, device="cuda", **kw) -> Composed:
    """Host or device transducers in, device result out."""
    if not isinstance(m1, DeviceFST):
        m1 = DeviceFST.from_host(m1, device)
    if not isinstance(m2, DeviceFST):
        m2 = DeviceFST.from_host(m2, device)
    return fstc_compose(m1, m2, **kw)


def compose_eps(m1, m2, eps: int, device="cuda", **kw) -> Composed:
    """Host or device transducers in, device result out (epsilon transitions)."""
    if not isinstance(m1, DeviceFST):
        m1 = DeviceFST.from_host(m1, device)
    if not isinstance(m2, DeviceFST):
        m2 = DeviceFST.from_host(m2, device)
    return fstc_compose_eps(m1, m2, eps, **kw)


def fstc_build_csr(m: DeviceFST, by_output: bool, stream=None) -> dict:
    """Device (state, inner symbol) layout of one transducer (fstc_build_csr)."""
    lib = load_library()
    dev = m.final.device
    n, nq = m.num_arcs, m.num_states
    out = {
        "row": torch.empty(nq + 1, dtype=torch.int32, device=dev),
        "seg_sym": torch.empty(max(n, 1), dtype=torch.int32, device=dev),
        "seg_off": torch.empty(n + 1, dtype=torch.int32, device=dev),
        "arc_part": torch.empty(max(n, 1), dtype=torch.int32, device=dev),
        "arc_weight": torch.empty(max(n, 1), dtype=torch.float32, device=dev),
        "part_base": torch.empty(nq + 1, dtype=torch.int32, device=dev),
        "part_target": torch.empty(max(n, 1), dtype=torch.int32, device=dev),
        "part_outer": torch.empty(max(n, 1), dtype=torch.int32, device=dev),
    }
    counts = np.zeros(3, np.uint64)
    s = m.struct()
    rc = lib.fstc_build_csr(ctypes.byref(s), 1 if by_output else 0, _stream_handle(stream),
                            *[out[k].data_ptr() for k in ("row", "seg_sym", "seg_off", "arc_part",
                                                          "arc_weight", "part_base", "part_target",
                                                          "part_outer")],
                            counts.ctypes.data)
    _check(rc)
    out["num_segments"], out["num_parts"], out["max_parts"] = (int(x) for x in counts)
    return out


def fstc_sort_pairs(keys: torch.Tensor, values: torch.Tensor, bit_lo: int = 0, bit_hi: int = 64,
                    stream=None):
    """In-place stable radix sort of int64 keys (as u64 bits) with int32 values."""
    assert keys.dtype == torch.int64 and values.dtype == torch.int32
    assert keys.is_contiguous() and values.is_contiguous() and keys.numel() == values.numel()
    _check(load_library().fstc_sort_pairs(keys.data_ptr(), values.data_ptr(), keys.numel(),
                                          bit_lo, bit_hi, _stream_handle(stream)))


def fstc_exclusive_scan_u64(x: torch.Tensor, stream=None) -> torch.Tensor:
    """Exclusive prefix sum of int64 (u64 bits) with the total appended."""
    assert x.dtype == torch.int64 and x.is_contiguous()
    out = torch.empty(x.numel() + 1, dtype=torch.int64, device=x.device)
    _check(load_library().fstc_exclusive_scan_u64(x.data_ptr() if x.numel() else None,
                                                  out.data_ptr(), x.numel(),
                                                  _stream_handle(stream)))
    return out


def fstc_exclusive_scan_u64_noalloc(x: torch.Tensor, out: torch.Tensor | None = None,
                                    stream=None) -> torch.Tensor:
    """The same scan through the entry point that allocates nothing (the
    library's per-device scratch array; n <= 2^28).  `out` (int64, n + 1
    elements) may be given so that the call needs no allocation at all."""
    assert x.dtype == torch.int64 and x.is_contiguous()
    if out is None:
        out = torch.empty(x.numel() + 1, dtype=torch.int64, device=x.device)
    assert out.dtype == torch.int64 and out.is_contiguous() and out.numel() >= x.numel() + 1
    _check(load_library().fstc_exclusive_scan_u64_noalloc(
        x.data_ptr() if x.numel() else None, out.data_ptr(), x.numel(), _stream_handle(stream)))
    return out
