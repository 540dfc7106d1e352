"""Shared test helpers: small CSR builders and comparisons (no method arithmetic
beyond what each test states explicitly)."""
import numpy as np
import scipy.sparse as sp

from paper_2608_09713_amd.workloads import CSR


def csr_from_dense(D, pattern=None, dtype=np.float64):
    """CSR of a dense array; ``pattern`` (bool) marks stored entries (may hold zeros)."""
    D = np.asarray(D)
    if pattern is None:
        pattern = D != 0
    m, n = D.shape
    rows, cols = np.nonzero(pattern)
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(np.bincount(rows, minlength=m), out=row_ptr[1:])
    return CSR(m, n, row_ptr, cols.astype(np.int32), D[rows, cols].astype(dtype))


def random_csr(rng, m, n, density, dtype=np.float64, signed=True, zeros=0.0):
    """Random canonical CSR; ``zeros`` is the fraction of stored entries set to 0."""
    pat = rng.random((m, n)) < density
    vals = rng.standard_normal((m, n)) if signed else rng.random((m, n)) + 0.5
    if zeros:
        vals[rng.random((m, n)) < zeros] = 0.0
    return csr_from_dense(np.where(pat, vals, 0.0), pattern=pat, dtype=dtype)


def to_scipy(A, values=None):
    v = A.values if values is None else values
    if v is None:
        v = np.ones(len(A.col_idx))
    return sp.csr_matrix((v, A.col_idx, A.row_ptr), shape=(A.nrows, A.ncols))


def dense_of(A):
    D = np.zeros((A.nrows, A.ncols))
    P = np.zeros((A.nrows, A.ncols), dtype=bool)
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    v = A.values if A.values is not None else np.ones(len(A.col_idx))
    D[rows, A.col_idx] = v
    P[rows, A.col_idx] = True
    return D, P


def result_to_dense(R, ncols):
    D = np.zeros((R.nrows, ncols))
    P = np.zeros((R.nrows, ncols), dtype=bool)
    rows = np.repeat(np.arange(R.nrows), np.diff(R.row_ptr))
    D[rows, R.col_idx] = R.values
    P[rows, R.col_idx] = True
    return D, P


def assert_canonical_rows(row_ptr, col_idx):
    for i in range(len(row_ptr) - 1):
        seg = col_idx[row_ptr[i]:row_ptr[i + 1]]
        assert np.all(np.diff(seg) > 0), f"row {i} not strictly increasing"
