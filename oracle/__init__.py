"""CPU oracle for tril(A A^T), the off-diagonal block A_i A_j^T and the mirror.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg use it to check and time the GPU library.  The
library never imports, links or calls anything here, and this package imports
nothing from the library.

The arithmetic lives in ``spsyrk_oracle.cpp`` (single-threaded Gustavson with
an ordered-map accumulator, written from the definition C = A A^T of Sec. II-A,
the lower-triangle restriction of Sec. III-A and the symmetric completion
C = C_L + C_L^T - D of Eq. (spmv)); a thin driver there runs the same per-row
code on several threads, for timing and for checking large results.  This
module only marshals numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spsyrk_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

SEMIRINGS = {"f64": 0, "f32": 1, "count": 2, "jaccard": 3}
_OUT_DTYPE = {0: np.float64, 1: np.float32, 2: np.int32, 3: np.float32}


def build(force: bool = False) -> str:
    """Compile the oracle with g++ (host only)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(out_path: str) -> str:
    """Compile the same source with AddressSanitizer and UndefinedBehaviorSanitizer
    into ``out_path`` (host code only; the tests load it in a child process
    with the ASan runtime preloaded and pass it as ``lib=`` to every entry point)."""
    subprocess.check_call(["g++", "-O1", "-g", "-std=c++17", "-shared", "-fPIC", "-pthread",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-o", out_path, _SRC])
    return out_path


def _declare(lib):
    i64, i32p, i64p, vp = ctypes.c_int64, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p
    lib.oracle_syrk.argtypes = [ctypes.c_int, ctypes.c_int, i64, i64, i64p, i32p, vp,
                                i64, i64, i64p, i32p, vp, i64p, i64, ctypes.POINTER(vp)]
    lib.oracle_syrk.restype = ctypes.c_int
    lib.oracle_syrk_threads.argtypes = lib.oracle_syrk.argtypes[:-1] + [ctypes.c_int, ctypes.POINTER(vp)]
    lib.oracle_syrk_threads.restype = ctypes.c_int
    lib.oracle_mirror.argtypes = [i64, i64p, i32p, vp, ctypes.c_int, ctypes.POINTER(vp)]
    lib.oracle_mirror.restype = ctypes.c_int
    lib.oracle_check_canonical.argtypes = [i64, i64, i64p, i32p]
    lib.oracle_check_canonical.restype = ctypes.c_int
    lib.oracle_result_nrows.argtypes = [vp]
    lib.oracle_result_nrows.restype = i64
    lib.oracle_result_nnz.argtypes = [vp]
    lib.oracle_result_nnz.restype = i64
    lib.oracle_result_copy.argtypes = [vp, i64p, i32p, vp, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_uint32)]
    lib.oracle_result_copy.restype = None
    lib.oracle_result_free.argtypes = [vp]
    lib.oracle_result_free.restype = None
    return lib


def _load(path: Optional[str] = None):
    """The oracle library; ``path`` loads another build of the same source
    (the tests plant mistakes in copies of it to check that the pins fail)."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    with _lock:
        if _lib is None:
            build()
            _lib = _declare(ctypes.CDLL(_LIB))
    return _lib


class OracleError(RuntimeError):
    pass


@dataclass
class Result:
    nrows: int
    ncols: int
    row_ptr: np.ndarray
    col_idx: np.ndarray
    values: np.ndarray
    sum_abs: Optional[np.ndarray] = None   # sum of |a_ik a_jk| per entry (fp tolerance scale)
    count: Optional[np.ndarray] = None     # number of shared columns per entry

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])


def _p(a, t):
    return a.ctypes.data_as(ctypes.POINTER(t)) if a is not None else None


def _csr_args(A, semiring):
    rp = np.ascontiguousarray(A.row_ptr, dtype=np.int64)
    ci = np.ascontiguousarray(A.col_idx, dtype=np.int32)
    if semiring == 0:
        v = np.ascontiguousarray(A.values, dtype=np.float64)
    elif semiring == 1:
        v = np.ascontiguousarray(A.values, dtype=np.float32)
    else:
        v = None
    return rp, ci, v


def _take(lib, h, sr, nrows, ncols, with_aux=True) -> Result:
    try:
        nnz = lib.oracle_result_nnz(h)
        rp = np.empty(nrows + 1, dtype=np.int64)
        ci = np.empty(nnz, dtype=np.int32)
        val = np.empty(nnz, dtype=_OUT_DTYPE[sr])
        sa = np.empty(nnz, dtype=np.float64) if with_aux else None
        cnt = np.empty(nnz, dtype=np.uint32) if with_aux else None
        lib.oracle_result_copy(h, _p(rp, ctypes.c_int64), _p(ci, ctypes.c_int32),
                               val.ctypes.data_as(ctypes.c_void_p), sr, 0,
                               _p(sa, ctypes.c_double), _p(cnt, ctypes.c_uint32))
    finally:
        lib.oracle_result_free(h)
    return Result(nrows, ncols, rp, ci, val, sa, cnt)


def _run(mode, A, B, semiring, rows, lib=None, threads=1):
    lib = lib or _load()
    sr = SEMIRINGS[semiring] if isinstance(semiring, str) else int(semiring)
    rp, ci, v = _csr_args(A, sr)
    if B is not None:
        rpb, cib, vb = _csr_args(B, sr)
        mb, nb = B.nrows, B.ncols
    else:
        rpb = cib = vb = None
        mb = nb = 0
    sel = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    h = ctypes.c_void_p()
    args = (mode, sr, A.nrows, A.ncols, _p(rp, ctypes.c_int64), _p(ci, ctypes.c_int32),
            v.ctypes.data_as(ctypes.c_void_p) if v is not None else None,
            mb, nb, _p(rpb, ctypes.c_int64), _p(cib, ctypes.c_int32),
            vb.ctypes.data_as(ctypes.c_void_p) if vb is not None else None,
            _p(sel, ctypes.c_int64), 0 if sel is None else len(sel))
    if threads > 1:
        rc = lib.oracle_syrk_threads(*args, int(threads), ctypes.byref(h))
    else:
        rc = lib.oracle_syrk(*args, ctypes.byref(h))
    if rc != 0:
        raise OracleError({1: "input not canonical", 2: "shape mismatch", 3: "out of memory"}.get(rc, str(rc)))
    nrows = A.nrows if sel is None else len(sel)
    return _take(lib, h, sr, nrows, A.nrows if B is None else B.nrows)


def lower(A, semiring, rows=None, lib=None, threads=1) -> Result:
    """C_L = tril(A A^T) (diagonal included); ``rows`` restricts to a row
    subset; ``threads`` > 1 computes blocks of rows on that many threads
    (the same rows through the same code, joined in order)."""
    return _run(0, A, None, semiring, rows, lib, threads)


def offdiag(Ai, Aj, semiring, rows=None, lib=None, threads=1) -> Result:
    """Rectangular C = A_i A_j^T with no triangle prune."""
    return _run(1, Ai, Aj, semiring, rows, lib, threads)


def host_threads() -> int:
    """Logical CPUs this process may run on (at most 16: the GPU machine's share)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def offdiag_half(Ai, Aj, half, semiring, lib=None) -> Result:
    """One half of the block C_ij = A_i A_j^T, as the two processes of a
    symmetric pair split it (Sec. III-A, Algorithm 3): ``"top"`` is rows
    [0, m_i // 2) of C_ij; ``"right"`` is columns [m_j // 2, m_j) of every row,
    with column ids in the block's numbering.  Written as the restriction of
    the full block to those rows or columns."""
    if half == "top":
        return offdiag(Ai, Aj, semiring, rows=np.arange(Ai.nrows // 2), lib=lib)
    if half != "right":
        raise ValueError(half)
    full = offdiag(Ai, Aj, semiring, lib=lib)
    keep = full.col_idx >= Aj.nrows // 2
    rows = np.repeat(np.arange(full.nrows), np.diff(full.row_ptr))
    rp = np.zeros(full.nrows + 1, dtype=np.int64)
    np.cumsum(np.bincount(rows[keep], minlength=full.nrows), out=rp[1:])
    return Result(full.nrows, full.ncols, rp, full.col_idx[keep], full.values[keep],
                  None if full.sum_abs is None else full.sum_abs[keep],
                  None if full.count is None else full.count[keep])


def mirror(m: int, row_ptr, col_idx, values, lib=None) -> Result:
    """Full symmetric CSR from the stored lower part (values copied bit for bit)."""
    lib = lib or _load()
    rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
    ci = np.ascontiguousarray(col_idx, dtype=np.int32)
    val = np.ascontiguousarray(values)
    nb = val.dtype.itemsize
    if nb not in (4, 8):
        raise ValueError("values must be 4- or 8-byte")
    h = ctypes.c_void_p()
    rc = lib.oracle_mirror(m, _p(rp, ctypes.c_int64), _p(ci, ctypes.c_int32),
                           val.ctypes.data_as(ctypes.c_void_p), nb, ctypes.byref(h))
    if rc != 0:
        raise OracleError("input not lower-triangular canonical CSR" if rc == 1 else str(rc))
    try:
        nnz = lib.oracle_result_nnz(h)
        out_rp = np.empty(m + 1, dtype=np.int64)
        out_ci = np.empty(nnz, dtype=np.int32)
        out_v = np.empty(nnz, dtype=val.dtype)
        lib.oracle_result_copy(h, _p(out_rp, ctypes.c_int64), _p(out_ci, ctypes.c_int32),
                               out_v.ctypes.data_as(ctypes.c_void_p), 4, nb, None, None)
    finally:
        lib.oracle_result_free(h)
    return Result(m, m, out_rp, out_ci, out_v)


def lower_accumulate(P: Result, A_s, semiring, lib=None) -> Result:
    """P + tril(A_s A_s^T) (Sec. III-A: a diagonal block is the sum over stages
    of SYRK(A_is)): the union of the two patterns, shared entries summed (fp64
    for f64, one float addition for f32, integers for count)."""
    T = lower(A_s, semiring, lib=lib)
    m = A_s.nrows
    rows_p = np.repeat(np.arange(m), np.diff(P.row_ptr))
    rows_t = np.repeat(np.arange(m), np.diff(T.row_ptr))
    keys = np.concatenate([rows_p * m + P.col_idx[: P.row_ptr[-1]], rows_t * m + T.col_idx])
    uk, inv = np.unique(keys, return_inverse=True)
    vals = np.concatenate([P.values[: P.row_ptr[-1]], T.values])
    if semiring == "count":
        out = np.zeros(len(uk), dtype=np.int64)
        np.add.at(out, inv, vals.astype(np.int64))
        out = out.astype(np.int32)
    else:
        out = np.zeros(len(uk), dtype=np.float64)
        np.add.at(out, inv, vals.astype(np.float64))
        out = out.astype(np.float32 if semiring == "f32" else np.float64)
    sa = None
    if T.sum_abs is not None:
        pa = P.sum_abs if P.sum_abs is not None else np.abs(P.values[: P.row_ptr[-1]].astype(np.float64))
        sa = np.zeros(len(uk))
        np.add.at(sa, inv, np.concatenate([pa, T.sum_abs]))
    rp = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(np.bincount(uk // m, minlength=m), out=rp[1:])
    return Result(m, m, rp, (uk % m).astype(np.int32), out, sa)


def symm(m: int, row_ptr, col_idx, values, X):
    """Y = C X for the symmetric C = C_L + C_L^T - D, from the stored lower
    part C_L (row_ptr, col_idx, values) as Eq. (spmv) writes it: the product
    with C_L, plus every strict-lower C_L(i, j) X(i, :) added to row j.  fp64.
    Returns (Y, S) with S = |C| |X| elementwise (the tolerance scale)."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    ci = np.asarray(col_idx, dtype=np.int64)[: rp[-1]]
    c = np.asarray(values)[: rp[-1]].astype(np.float64)
    X = np.asarray(X, dtype=np.float64).reshape(m, -1)
    rows = np.repeat(np.arange(m), np.diff(rp))
    Y = np.zeros_like(X)
    S = np.zeros_like(X)
    np.add.at(Y, rows, c[:, None] * X[ci])
    np.add.at(S, rows, np.abs(c[:, None] * X[ci]))
    off = ci != rows
    np.add.at(Y, ci[off], c[off, None] * X[rows[off]])
    np.add.at(S, ci[off], np.abs(c[off, None] * X[rows[off]]))
    return Y, S


def is_canonical(A) -> bool:
    lib = _load()
    rp = np.ascontiguousarray(A.row_ptr, dtype=np.int64)
    ci = np.ascontiguousarray(A.col_idx, dtype=np.int32)
    return lib.oracle_check_canonical(A.nrows, A.ncols, _p(rp, ctypes.c_int64), _p(ci, ctypes.c_int32)) == 0
