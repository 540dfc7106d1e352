"""Local sparse SYRK on one MI355X: tril(A A^T), A_i A_j^T and the mirror.

Thin binding over ``libspsyrk.so`` (C-ABI in ``include/spsyrk.h``).  This module
only marshals arguments: device memory and streams come from PyTorch, every
step of the computation runs in the library's HIP kernels, and a missing or
unloadable library raises instead of falling back to anything else.

    import torch, paper_2608_09713_amd as sp
    A = sp.DeviceCSR.from_host(csr, device="cuda:0")
    C = sp.lower(A, "jaccard")          # tril(A A^T), Jaccard values
    F = sp.mirror(C, "jaccard")         # full symmetric matrix
"""
from __future__ import annotations

import ctypes
import os
import threading
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspsyrk.so")
# SPSYRK_DEBUG=1 in the environment loads the build with the kernels' invariant
# checks (debug_flags() reads what they found); it must be set before the first call
DEBUG_LIB_PATH = os.path.join(_HERE, "libspsyrk_debug.so")

SEMIRINGS = {"f64": 0, "f32": 1, "count": 2, "jaccard": 3}
# dtype of A's values each semiring reads, and of the output values
_IN_DTYPE = {0: "float64", 1: "float32", 2: None, 3: None}
_OUT_DTYPE = {0: "float64", 1: "float32", 2: "int32", 3: "float32"}

STATUS = {0: "ok", 1: "invalid argument", 2: "not canonical", 3: "shape", 4: "out of memory",
          5: "overflow", 6: "hip error", 7: "too large for the fixed scratch"}


class SpsyrkError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"spsyrk: {STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class _Csr(ctypes.Structure):
    _fields_ = [("nrows", ctypes.c_int64), ("ncols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p), ("values", ctypes.c_void_p)]


class _CsrOut(ctypes.Structure):
    _fields_ = [("nrows", ctypes.c_int64), ("ncols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p), ("values", ctypes.c_void_p)]


_ALLOC = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t)
_FREE = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class _Allocator(ctypes.Structure):
    _fields_ = [("alloc", _ALLOC), ("free", _FREE), ("ctx", ctypes.c_void_p)]


class Stats(ctypes.Structure):
    _fields_ = [("nnz_out", ctypes.c_int64), ("csc_entries", ctypes.c_int64), ("heavy_rows", ctypes.c_int64),
                ("light_rows", ctypes.c_int64), ("products", ctypes.c_int64), ("heavy_entries", ctypes.c_int64),
                ("heavy_nnz_out", ctypes.c_int64), ("group_shift", ctypes.c_int32), ("row_bits", ctypes.c_int32),
                ("packed_staging", ctypes.c_int32), ("reserved", ctypes.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None
_lib_lock = threading.Lock()


def library():
    """The loaded C library; raises if it has not been built."""
    global _lib
    with _lib_lock:
        if _lib is None:
            # torch's HIP runtime comes up first: a process that loaded this
            # library before torch touched the device saw no device in it
            import torch
            torch.cuda.is_available()
            path = DEBUG_LIB_PATH if os.environ.get("SPSYRK_DEBUG") == "1" else LIB_PATH
            if not os.path.exists(path):
                raise ImportError(f"{path} is missing: run `python -m paper_2608_09713_amd.build` "
                                  "(or __graft_entry__.build()) first")
            lib = ctypes.CDLL(path)
            for name in ("spsyrk_lower", "spsyrk_offdiag", "spsyrk_offdiag_half", "spsyrk_mirror"):
                getattr(lib, name).restype = ctypes.c_int
            lib.spsyrk_lower.argtypes = [ctypes.POINTER(_Csr), ctypes.c_int, ctypes.POINTER(_Allocator),
                                         ctypes.c_void_p, ctypes.POINTER(_CsrOut)]
            lib.spsyrk_offdiag.argtypes = [ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), ctypes.c_int,
                                           ctypes.POINTER(_Allocator), ctypes.c_void_p, ctypes.POINTER(_CsrOut)]
            lib.spsyrk_offdiag_half.argtypes = [ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), ctypes.c_int,
                                                ctypes.c_int, ctypes.POINTER(_Allocator), ctypes.c_void_p,
                                                ctypes.POINTER(_CsrOut)]
            lib.spsyrk_mirror.argtypes = [ctypes.POINTER(_Csr), ctypes.c_int, ctypes.POINTER(_Allocator),
                                          ctypes.c_void_p, ctypes.POINTER(_CsrOut)]
            lib.spsyrk_lower_plan.restype = ctypes.c_int
            lib.spsyrk_lower_plan.argtypes = [ctypes.POINTER(_Csr), ctypes.c_int, ctypes.POINTER(_Allocator),
                                              ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p),
                                              ctypes.POINTER(_CsrOut)]
            lib.spsyrk_lower_execute.restype = ctypes.c_int
            lib.spsyrk_lower_execute.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(_Allocator),
                                                 ctypes.c_void_p, ctypes.POINTER(_CsrOut)]
            lib.spsyrk_plan_destroy.restype = ctypes.c_int
            lib.spsyrk_plan_destroy.argtypes = [ctypes.c_void_p]
            lib.spsyrk_lower_accumulate.restype = ctypes.c_int
            lib.spsyrk_lower_accumulate.argtypes = [ctypes.POINTER(_Csr), ctypes.POINTER(_Csr), ctypes.c_int,
                                                    ctypes.POINTER(_Allocator), ctypes.c_void_p,
                                                    ctypes.POINTER(_CsrOut)]
            lib.spsyrk_symm.restype = ctypes.c_int
            lib.spsyrk_symm.argtypes = [ctypes.POINTER(_Csr), ctypes.c_int, ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(_Allocator),
                                        ctypes.c_void_p]
            lib.spsyrk_symm_noalloc.restype = ctypes.c_int
            lib.spsyrk_symm_noalloc.argtypes = [ctypes.POINTER(_Csr), ctypes.c_int, ctypes.c_int64, ctypes.c_void_p,
                                                ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
            lib.spsyrk_status_string.argtypes = [ctypes.c_int]
            lib.spsyrk_status_string.restype = ctypes.c_char_p
            lib.spsyrk_last_error_detail.argtypes = []
            lib.spsyrk_last_error_detail.restype = ctypes.c_char_p
            lib.spsyrk_last_stats.argtypes = [ctypes.POINTER(Stats)]
            lib.spsyrk_last_stats.restype = ctypes.c_int
            lib.spsyrk_abi_version.restype = ctypes.c_int
            lib.spsyrk_timing_begin.restype = ctypes.c_int
            lib.spsyrk_timing_begin_phases.argtypes = [ctypes.c_uint32]
            lib.spsyrk_timing_begin_phases.restype = ctypes.c_int
            lib.spsyrk_timing_end.argtypes = [ctypes.POINTER(_PhaseTimes)]
            lib.spsyrk_timing_end.restype = ctypes.c_int
            lib.spsyrk_debug_build.argtypes = []
            lib.spsyrk_debug_build.restype = ctypes.c_int
            lib.spsyrk_debug_flags.argtypes = [ctypes.POINTER(ctypes.c_uint32)]
            lib.spsyrk_debug_flags.restype = ctypes.c_int
            _lib = lib
    return _lib


EXPORTS = ("spsyrk_lower", "spsyrk_lower_plan", "spsyrk_lower_execute", "spsyrk_plan_destroy",
           "spsyrk_lower_accumulate", "spsyrk_offdiag", "spsyrk_offdiag_half", "spsyrk_mirror",
           "spsyrk_symm", "spsyrk_symm_noalloc",
           "spsyrk_status_string",
           "spsyrk_last_error_detail", "spsyrk_last_stats", "spsyrk_abi_version", "spsyrk_timing_begin",
           "spsyrk_timing_begin_phases", "spsyrk_timing_end", "spsyrk_debug_build", "spsyrk_debug_flags")


def debug_build() -> bool:
    """Whether the loaded library has the kernels' invariant checks compiled in."""
    return bool(library().spsyrk_debug_build())


def debug_flags() -> int:
    """Waits for the device, then returns and clears the OR of the check bits
    that the debug build's kernels raised (0 in the ordinary build)."""
    lib = library()
    f = ctypes.c_uint32(0)
    rc = lib.spsyrk_debug_flags(ctypes.byref(f))
    if rc != 0:
        raise SpsyrkError(rc, lib.spsyrk_last_error_detail().decode())
    return int(f.value)

PHASES = ("validate", "colindex", "light_symbolic", "heavy_symbolic", "scan", "light_numeric", "heavy_numeric",
          "mirror_count", "mirror_copy", "mirror_transpose", "runs", "compact", "colindex_passes", "colindex_pack")


class _PhaseTimes(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * len(PHASES)), ("launches", ctypes.c_int64 * len(PHASES))]


@dataclass
class DeviceCSR:
    """CSR whose arrays are torch tensors on one GPU."""
    nrows: int
    ncols: int
    row_ptr: "object"            # torch.int64 [nrows + 1]
    col_idx: "object"            # torch.int32 [>= nnz]
    values: "object" = None      # torch tensor [>= nnz] or None
    nnz: Optional[int] = None

    def __post_init__(self):
        if self.nnz is None:
            self.nnz = int(self.row_ptr[-1].item()) if self.nrows >= 0 and self.row_ptr.numel() else 0

    @staticmethod
    def from_host(A, device="cuda:0", value_dtype=None) -> "DeviceCSR":
        """Upload a host CSR (any object with nrows, ncols, row_ptr, col_idx, values)."""
        import torch
        rp = torch.from_numpy(np.ascontiguousarray(A.row_ptr, dtype=np.int64)).to(device)
        ci = torch.from_numpy(np.ascontiguousarray(A.col_idx, dtype=np.int32)).to(device)
        v = None
        if A.values is not None:
            vals = np.ascontiguousarray(A.values)
            if value_dtype is not None:
                vals = vals.astype(value_dtype)
            v = torch.from_numpy(vals).to(device)
        return DeviceCSR(A.nrows, A.ncols, rp, ci, v, int(A.row_ptr[-1]) if len(A.row_ptr) else 0)

    def to_host(self):
        """(row_ptr, col_idx, values) as numpy arrays of exactly nnz entries."""
        rp = self.row_ptr.cpu().numpy()
        ci = self.col_idx[: self.nnz].cpu().numpy()
        v = self.values[: self.nnz].cpu().numpy() if self.values is not None else None
        return rp, ci, v


class _TorchArena:
    """Device allocations for one call, backed by torch's caching allocator on
    the call's stream.  Pointers handed to the library map to their tensors."""

    def __init__(self, device):
        import torch
        self.torch = torch
        self.device = device
        self.live = {}
        self._alloc = _ALLOC(self._do_alloc)
        self._free = _FREE(self._do_free)
        self.struct = _Allocator(self._alloc, self._free, None)

    def _do_alloc(self, ctx, nbytes):
        try:
            t = self.torch.empty(int(nbytes), dtype=self.torch.uint8, device=self.device)
        except Exception:  # out of memory: report NULL, the library returns SPSYRK_ERR_OOM
            return None
        p = t.data_ptr()
        self.live[p] = t
        return p

    def _do_free(self, ctx, p):
        self.live.pop(p, None)

    def take(self, p, dtype, count):
        if not p:
            return None
        t = self.live.pop(p)
        return t.view(dtype)[:count] if count > 0 else t.view(dtype)[:0]


def _csr_struct(A: DeviceCSR, sr: int, need_values: bool):
    import torch
    if A.row_ptr.dtype != torch.int64 or A.col_idx.dtype != torch.int32:
        raise TypeError("row_ptr must be int64 and col_idx int32")
    for t in (A.row_ptr, A.col_idx):
        if not t.is_cuda or not t.is_contiguous():
            raise TypeError("CSR arrays must be contiguous device tensors")
    vp = None
    if need_values and _IN_DTYPE[sr] is not None:
        if A.values is None:
            raise TypeError("values are required for plus-times semirings")
        want = getattr(torch, _IN_DTYPE[sr])
        if A.values.dtype != want or not A.values.is_contiguous():
            raise TypeError(f"values must be a contiguous {want} tensor")
        vp = A.values.data_ptr()
    elif not need_values and A.values is not None:
        vp = A.values.data_ptr()
    return _Csr(A.nrows, A.ncols, A.nnz, A.row_ptr.data_ptr(), A.col_idx.data_ptr() if A.col_idx.numel() else 0, vp)


def _sr(semiring) -> int:
    return SEMIRINGS[semiring] if isinstance(semiring, str) else int(semiring)


def _take_out(arena, out, sr):
    import torch
    odt = getattr(torch, _OUT_DTYPE[sr])
    rp = arena.take(out.row_ptr, torch.int64, out.nrows + 1)
    ci = arena.take(out.col_idx, torch.int32, out.nnz)
    v = arena.take(out.values, odt, out.nnz) if out.values else None
    return DeviceCSR(out.nrows, out.ncols, rp, ci, v, out.nnz)


def _call(fn_name, args, sr, device, out_has_values=True):
    import torch
    lib = library()
    arena = _TorchArena(device)
    out = _CsrOut()
    stream = torch.cuda.current_stream(device).cuda_stream
    rc = getattr(lib, fn_name)(*args(arena), ctypes.c_void_p(stream), ctypes.byref(out))
    if rc != 0:
        raise SpsyrkError(rc, lib.spsyrk_last_error_detail().decode())
    C = _take_out(arena, out, sr)
    if arena.live:
        raise RuntimeError("library left allocations unreleased")
    return C


class Plan:
    """A lower product's pattern-only results kept on the device
    (spsyrk_lower_plan); ``execute(values)`` recomputes C_L for new values of
    the same pattern (spsyrk_lower_execute).  ``close()`` (or garbage
    collection) releases the plan (spsyrk_plan_destroy)."""

    def __init__(self, handle, arena, sr, nnz, device):
        self._h = handle
        self._arena = arena  # owns the plan's device buffers
        self.sr = sr
        self.nnz = nnz
        self.device = device

    def execute(self, values=None) -> DeviceCSR:
        import torch
        if self._h is None:
            raise RuntimeError("plan is closed")
        vp = None
        if _IN_DTYPE[self.sr] is not None:
            want = getattr(torch, _IN_DTYPE[self.sr])
            if values is None or values.dtype != want or not values.is_contiguous() or values.numel() < self.nnz:
                raise TypeError(f"values must be a contiguous {want} tensor of {self.nnz} entries")
            vp = values.data_ptr()
        return _call("spsyrk_lower_execute",
                     lambda ar: (self._h, ctypes.c_void_p(vp), ctypes.byref(ar.struct)), self.sr, self.device)

    def close(self):
        if self._h is not None:
            library().spsyrk_plan_destroy(self._h)
            self._h = None
            if self._arena.live:
                raise RuntimeError("plan buffers left unreleased")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def lower_plan(A: DeviceCSR, semiring="f64"):
    """(plan, C_L): C_L = tril(A A^T) and a plan for new values of A's pattern
    (spsyrk_lower_plan)."""
    import torch
    sr = _sr(semiring)
    lib = library()
    a = _csr_struct(A, sr, True)
    dev = A.row_ptr.device
    arena = _TorchArena(dev)
    out = _CsrOut()
    h = ctypes.c_void_p()
    stream = torch.cuda.current_stream(dev).cuda_stream
    rc = lib.spsyrk_lower_plan(ctypes.byref(a), sr, ctypes.byref(arena.struct), ctypes.c_void_p(stream),
                               ctypes.byref(h), ctypes.byref(out))
    if rc != 0:
        raise SpsyrkError(rc, lib.spsyrk_last_error_detail().decode())
    C = _take_out(arena, out, sr)
    return Plan(h, arena, sr, A.nnz, dev), C


def lower(A: DeviceCSR, semiring="f64") -> DeviceCSR:
    """C_L = tril(A A^T) with the diagonal (spsyrk_lower)."""
    sr = _sr(semiring)
    a = _csr_struct(A, sr, True)
    return _call("spsyrk_lower", lambda ar: (ctypes.byref(a), sr, ctypes.byref(ar.struct)), sr, A.row_ptr.device)


def lower_accumulate(C_prev: DeviceCSR, A_s: DeviceCSR, semiring="f64") -> DeviceCSR:
    """C_prev + tril(A_s A_s^T), one stage added to an accumulated lower part
    (spsyrk_lower_accumulate; f64, f32 or count)."""
    sr = _sr(semiring)
    p = _csr_struct(C_prev, sr, False)
    a = _csr_struct(A_s, sr, True)
    return _call("spsyrk_lower_accumulate", lambda ar: (ctypes.byref(p), ctypes.byref(a), sr, ctypes.byref(ar.struct)),
                 sr, A_s.row_ptr.device)


def offdiag(Ai: DeviceCSR, Aj: DeviceCSR, semiring="f64") -> DeviceCSR:
    """C = A_i A_j^T, full rectangular block (spsyrk_offdiag)."""
    sr = _sr(semiring)
    a = _csr_struct(Ai, sr, True)
    b = _csr_struct(Aj, sr, True)
    return _call("spsyrk_offdiag", lambda ar: (ctypes.byref(a), ctypes.byref(b), sr, ctypes.byref(ar.struct)),
                 sr, Ai.row_ptr.device)


HALVES = {"top": 0, "right": 1}


def offdiag_half(Ai: DeviceCSR, Aj: DeviceCSR, half: str, semiring="f64") -> DeviceCSR:
    """One half of C = A_i A_j^T (spsyrk_offdiag_half): ``half="top"`` gives rows
    [0, m_i // 2); ``half="right"`` gives columns [m_j // 2, m_j) of every row,
    with column ids in the block's numbering."""
    sr = _sr(semiring)
    h = HALVES[half]
    a = _csr_struct(Ai, sr, True)
    b = _csr_struct(Aj, sr, True)
    return _call("spsyrk_offdiag_half",
                 lambda ar: (ctypes.byref(a), ctypes.byref(b), h, sr, ctypes.byref(ar.struct)), sr,
                 Ai.row_ptr.device)


def symm(C_lower: DeviceCSR, X, semiring="f64"):
    """Y = C X with C = C_L + C_L^T - D from the stored lower part only
    (spsyrk_symm).  X: a device tensor of m or m x k (row-major rows may be
    padded: its stride is passed as the leading dimension), float64 for the
    f64 and count semirings, float32 for f32 and jaccard.  Returns Y shaped
    like X (contiguous)."""
    import torch
    sr = _sr(semiring)
    want = torch.float64 if sr in (0, 2) else torch.float32
    if X.dtype != want:
        raise TypeError(f"X must be {want} for semiring {semiring}")
    X2 = X.unsqueeze(1) if X.dim() == 1 else X
    if X2.dim() != 2 or X2.shape[0] != C_lower.nrows or X2.stride(1) != 1:
        raise ValueError("X must be m or m x k with unit column stride")
    m, k = X2.shape
    Y2 = torch.empty((m, k), dtype=want, device=X.device)
    lib = library()
    arena = _TorchArena(X.device)
    a = _csr_struct(C_lower, sr, False)
    stream = torch.cuda.current_stream(X.device).cuda_stream
    rc = lib.spsyrk_symm(ctypes.byref(a), sr, k, ctypes.c_void_p(X2.data_ptr()), X2.stride(0),
                         ctypes.c_void_p(Y2.data_ptr()), k, ctypes.byref(arena.struct), ctypes.c_void_p(stream))
    if rc != 0:
        raise SpsyrkError(rc, lib.spsyrk_last_error_detail().decode())
    if arena.live:
        raise RuntimeError("library left allocations unreleased")
    return Y2.squeeze(1) if X.dim() == 1 else Y2


def symm_noalloc(C_lower: DeviceCSR, X, Y=None, semiring="f64"):
    """Y = C X as ``symm`` does, through spsyrk_symm_noalloc: the library
    allocates nothing (its workspace is a fixed per-device array, so calls on
    one device must not overlap).  ``Y``: an optional preallocated output
    shaped like X (m or m x k, unit column stride); returns Y."""
    import torch
    sr = _sr(semiring)
    want = torch.float64 if sr in (0, 2) else torch.float32
    if X.dtype != want:
        raise TypeError(f"X must be {want} for semiring {semiring}")
    X2 = X.unsqueeze(1) if X.dim() == 1 else X
    if X2.dim() != 2 or X2.shape[0] != C_lower.nrows or X2.stride(1) != 1:
        raise ValueError("X must be m or m x k with unit column stride")
    m, k = X2.shape
    if Y is None:
        Y = torch.empty(X.shape, dtype=want, device=X.device)
    Y2 = Y.unsqueeze(1) if Y.dim() == 1 else Y
    if Y2.dtype != want or tuple(Y2.shape) != (m, k) or Y2.stride(1) != 1:
        raise ValueError("Y must match X's shape and dtype with unit column stride")
    lib = library()
    a = _csr_struct(C_lower, sr, False)
    stream = torch.cuda.current_stream(X.device).cuda_stream
    rc = lib.spsyrk_symm_noalloc(ctypes.byref(a), sr, k, ctypes.c_void_p(X2.data_ptr()), X2.stride(0),
                                 ctypes.c_void_p(Y2.data_ptr()), Y2.stride(0), ctypes.c_void_p(stream))
    if rc != 0:
        raise SpsyrkError(rc, lib.spsyrk_last_error_detail().decode())
    return Y


def mirror(C_lower: DeviceCSR, semiring="f64") -> DeviceCSR:
    """C = C_L + C_L^T - D from a stored lower part (spsyrk_mirror)."""
    import torch
    sr = _sr(semiring)
    a = _csr_struct(C_lower, sr, False)
    C = _call("spsyrk_mirror", lambda ar: (ctypes.byref(a), sr, ctypes.byref(ar.struct)), sr,
              C_lower.row_ptr.device)
    if C.values is None and C_lower.values is not None:
        # an empty C_L's values reach the library as a null pointer (a pattern
        # without values); its mirror still has (no) values of the output type
        C.values = torch.empty(0, dtype=getattr(torch, _OUT_DTYPE[sr]), device=C_lower.row_ptr.device)
    return C


def stats() -> dict:
    """Counters of the last successful call on this thread."""
    s = Stats()
    library().spsyrk_last_stats(ctypes.byref(s))
    return s.as_dict()


def timing_begin(phases=None) -> None:
    """Start recording HIP events around every phase of the calls on this
    thread, or around the named phases only."""
    if phases is None:
        library().spsyrk_timing_begin()
    else:
        mask = 0
        for name in phases:
            mask |= 1 << PHASES.index(name)
        library().spsyrk_timing_begin_phases(mask)


def timing_end() -> dict:
    """Stop recording; {phase: (summed ms, timed launches)} for the phases seen."""
    t = _PhaseTimes()
    rc = library().spsyrk_timing_end(ctypes.byref(t))
    if rc != 0:
        raise SpsyrkError(rc, library().spsyrk_last_error_detail().decode())
    return {name: (t.ms[k], t.launches[k]) for k, name in enumerate(PHASES) if t.launches[k]}
