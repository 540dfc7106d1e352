"""Seeded generators: determinism, canonical CSR and the stated statistics."""
import numpy as np
import pytest

from paper_2608_09713_amd import workloads as W
import oracle


@pytest.mark.parametrize("name,shift", [("tiny_uniform_f64", 0), ("kmer_i32", 7), ("rmat20_f32", 8),
                                        ("offdiag_f64", 7), ("jaccard_large", 9)])
def test_deterministic_and_canonical(name, shift):
    a = W.make(name, 1, shift)
    b = W.make(name, 1, shift)
    for key in ("A", "B"):
        if key not in a:
            continue
        X, Y = a[key], b[key]
        np.testing.assert_array_equal(X.row_ptr, Y.row_ptr)
        np.testing.assert_array_equal(X.col_idx, Y.col_idx)
        if X.values is not None:
            np.testing.assert_array_equal(X.values, Y.values)
        assert X.row_ptr.dtype == np.int64 and X.col_idx.dtype == np.int32
        assert oracle.is_canonical(X)
    c = W.make(name, 2, shift)["A"]
    assert not (c.nnz == a["A"].nnz and np.array_equal(c.col_idx, a["A"].col_idx))


def test_tiny_shape():
    A = W.make("tiny_uniform_f64")["A"]
    assert (A.nrows, A.ncols, A.nnz) == (4096, 16384, 32768)
    assert np.all(np.diff(A.row_ptr) == 8)
    assert np.all((A.values > 0) & (A.values <= 1))


def test_kmer_filter_and_row_lengths():
    A = W.make("kmer_i32", 1, 6)["A"]
    cnt = np.bincount(A.col_idx, minlength=A.ncols)
    assert cnt.max() <= 50
    assert np.diff(A.row_ptr).max() <= 32
    assert A.values is None


def test_rmat_no_loops_no_duplicates():
    A = W.make("rmat20_f32", 1, 8)["A"]
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    assert not np.any(rows == A.col_idx)
    key = rows.astype(np.int64) * A.ncols + A.col_idx
    assert len(np.unique(key)) == len(key)
    assert A.values.dtype == np.float32 and np.all((A.values > 0) & (A.values <= 1))


def test_bounded_zipf_matches_pmf():
    z = W.BoundedZipf(30, 0.9)
    x = z.sample(W.rng_for(7), 1_000_000)
    p = np.arange(1, 31) ** -0.9
    p /= p.sum()
    f = np.bincount(x, minlength=31)[1:] / len(x)
    assert x.min() >= 1 and x.max() <= 30
    assert np.abs(f - p).max() < 3e-3
