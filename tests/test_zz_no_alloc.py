"""The allocation-free product from a stored lower part (spsyrk_symm_noalloc)
against the allocating one (spsyrk_symm) through the C-ABI: two calls in a
row on the same device, the second with a smaller input (the shared scratch
keeps the first call's contents), for the four semirings; one call in the
range where spsyrk_symm takes its bucketed path; and the size limit."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2608_09713_amd as sp
from paper_2608_09713_amd.workloads import CSR
from tests.helpers import random_csr

pytestmark = pytest.mark.gpu

VDT = {"f64": np.float64, "f32": np.float32, "count": None, "jaccard": None}
SYMM_TOL = {"f64": 1e-12, "count": 1e-12, "jaccard": 2.0 ** -24, "f32": 1e-5 + 2.0 ** -24}


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available()
    sp.library()
    return "cuda:0"


def _scale(L, X):
    # sum over the terms of |C_L entry scale| |x| (the product's tolerance scale)
    ent = L.sum_abs if L.sum_abs is not None else np.abs(L.values.astype(np.float64))
    s, _ = oracle.symm(L.nrows, L.row_ptr, L.col_idx, ent, np.abs(X))
    return s


def _sparse_rows(rng, m, n, per_row):
    # up to per_row distinct uniform columns per row, drawn without a dense array
    cols = np.sort(rng.integers(0, n, size=(m, per_row)), axis=1)
    keep = np.ones(cols.shape, dtype=bool)
    keep[:, 1:] = cols[:, 1:] != cols[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(keep.sum(axis=1), out=rp[1:])
    ci = cols[keep].astype(np.int32)
    return CSR(m, n, rp, ci, rng.standard_normal(len(ci)))


def _case(dev, rng, semiring, m, n, density, k):
    import torch
    vdt = VDT[semiring]
    xdt = np.float64 if semiring in ("f64", "count") else np.float32
    if density < 1e-3:
        A = _sparse_rows(rng, m, n, max(1, int(round(density * n))))
    else:
        A = random_csr(rng, m, n, density, signed=True)
    Ah = A.with_values(A.values.astype(vdt) if vdt is not None else None)
    dA = sp.DeviceCSR.from_host(Ah, dev)
    C = sp.lower(dA, semiring)
    L = oracle.lower(Ah, semiring)
    X = rng.standard_normal((m, k + 1)).astype(xdt)
    Xd = torch.from_numpy(X).to(dev)[:, :k]
    return C, L, X[:, :k].astype(np.float64), Xd


def _check(Y, Yref, scale, semiring, what):
    err = np.abs(Y.astype(np.float64) - Yref.astype(np.float64))
    bad = err > SYMM_TOL[semiring] * np.maximum(scale, np.abs(Yref)) + 1e-300
    assert not bad.any(), f"{what}: {int(bad.sum())} elements out of tolerance, max err {float(err.max())!r}"


@pytest.mark.parametrize("semiring", ["f64", "f32", "count", "jaccard"])
def test_noalloc_matches_symm_twice(dev, semiring):
    import torch
    rng = np.random.default_rng(71)
    for call, (m, n, dens, k) in enumerate(((3000, 2500, 0.004, 3), (700, 900, 0.01, 1))):
        print(f"[symm_noalloc {semiring}] call {call}: m={m} k={k}", flush=True)
        C, L, X, Xd = _case(dev, rng, semiring, m, n, dens, k)
        Yref = sp.symm(C, Xd, semiring).cpu().numpy()
        Y = torch.full((m, k), float("nan"), dtype=Xd.dtype, device=dev)
        sp.symm_noalloc(C, Xd, Y, semiring)
        _check(Y.cpu().numpy(), Yref, _scale(L, X), semiring, f"call {call}")


def test_noalloc_where_symm_takes_buckets(dev):
    # 2^19 + 3000 rows and one column: spsyrk_symm sums the transposed term
    # through buckets, the allocation-free call with atomic adds
    import torch
    rng = np.random.default_rng(72)
    m = (1 << 19) + 3000
    C, L, X, Xd = _case(dev, rng, "f64", m, 1 << 20, 4 / float(1 << 20), 1)
    print(f"[symm_noalloc buckets] m={m} nnz_L={L.nnz}", flush=True)
    Yref = sp.symm(C, Xd, "f64").cpu().numpy()
    Y = sp.symm_noalloc(C, Xd, None, "f64").cpu().numpy()
    _check(Y, Yref, _scale(L, X), "f64", "bucketed range")


def test_noalloc_rejects_oversize(dev):
    # m k = 2^21 * 9 doubles exceed the fixed scratch: refused before any
    # device work, and the next call still works
    import torch
    lib = sp.library()
    m = 1 << 21
    rp = torch.zeros(m + 1, dtype=torch.int64, device=dev)
    ci = torch.zeros(1, dtype=torch.int32, device=dev)
    X = torch.zeros((m, 9), dtype=torch.float64, device=dev)
    a = sp._Csr(m, m, 0, rp.data_ptr(), ci.data_ptr(), None)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    rc = lib.spsyrk_symm_noalloc(ctypes.byref(a), 0, 9, ctypes.c_void_p(X.data_ptr()), 9,
                                 ctypes.c_void_p(X.data_ptr()), 9, s)
    assert rc == 7, lib.spsyrk_last_error_detail()
    assert b"scratch" in lib.spsyrk_last_error_detail()
    rng = np.random.default_rng(73)
    C, L, X, Xd = _case(dev, rng, "f64", 500, 600, 0.02, 2)
    Y = sp.symm_noalloc(C, Xd, None, "f64").cpu().numpy()
    ref, _ = oracle.symm(L.nrows, L.row_ptr, L.col_idx, L.values, X)
    _check(Y, ref, _scale(L, X), "f64", "after a refused call")
