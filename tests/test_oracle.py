"""Pins of the CPU oracle against things other than itself.

Every check here is independent of the oracle's own code: hand-worked values
(tests/golden), dense brute force with numpy, scipy.sparse products, closed
forms (F_L = sum_k c_k (c_k + 1) / 2), exact invariants (symmetry, diagonal =
row squared norms, C = C_L + C_L^T - D) and special cases.  A final group
plants mistakes in copies of the oracle source and checks that the pins fail.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from paper_2608_09713_amd import workloads as W
from paper_2608_09713_amd.workloads import CSR
from tests.helpers import (assert_canonical_rows, csr_from_dense, dense_of, random_csr,
                           result_to_dense, to_scipy)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_small.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _csr(g, values=True):
    v = np.array(g["values"], dtype=np.float64) if values and "values" in g else None
    return CSR(g["nrows"], g["ncols"], np.array(g["row_ptr"], dtype=np.int64),
               np.array(g["col_idx"], dtype=np.int32), v)


# --------------------------------------------------------------------------
# hand-worked fixtures (Sec. II-A definition, Sec. III-A lower part, Eq. (spmv))


def check_golden(lib=None):
    g = _golden()
    P = _csr(g["P"])
    R = oracle.lower(P, "f64", lib=lib)
    e = g["P"]["lower_f64"]
    np.testing.assert_array_equal(R.row_ptr, e["row_ptr"])
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values, e["values"])

    R = oracle.lower(P.with_values(None), "count", lib=lib)
    e = g["P"]["lower_count"]
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values, e["values"])

    R = oracle.lower(P.with_values(None), "jaccard", lib=lib)
    e = g["P"]["lower_jaccard"]
    want = np.float32(e["numerator"]) / np.float32(e["denominator"])
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values.view(np.uint32), want.view(np.uint32))

    R = oracle.lower(P, "f64", lib=lib)
    M = oracle.mirror(P.nrows, R.row_ptr, R.col_idx, R.values, lib=lib)
    e = g["P"]["mirror_f64"]
    np.testing.assert_array_equal(M.row_ptr, e["row_ptr"])
    np.testing.assert_array_equal(M.col_idx, e["col_idx"])
    np.testing.assert_array_equal(M.values, e["values"])

    Ai = CSR(2, 5, P.row_ptr[:3].copy(), P.col_idx[:4], P.values[:4])
    Aj = CSR(2, 5, P.row_ptr[2:] - P.row_ptr[2], P.col_idx[4:], P.values[4:])
    R = oracle.offdiag(Ai, Aj, "f64", lib=lib)
    e = g["P"]["offdiag_rows01_by_rows23_f64"]
    np.testing.assert_array_equal(R.row_ptr, e["row_ptr"])
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values, e["values"])

    Q = _csr(g["Q"])
    R = oracle.lower(Q, "f64", lib=lib)
    e = g["Q"]["lower_f64"]
    np.testing.assert_array_equal(R.row_ptr, e["row_ptr"])
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values, e["values"])
    R = oracle.lower(Q.with_values(None), "count", lib=lib)
    np.testing.assert_array_equal(R.values, g["Q"]["lower_count"]["values"])

    J = _csr(g["jaccard_pair"], values=False)
    R = oracle.lower(J, "jaccard", lib=lib)
    e = g["jaccard_pair"]["lower_jaccard"]
    np.testing.assert_array_equal(R.col_idx, e["col_idx"])
    np.testing.assert_array_equal(R.values, np.float32(e["values"]))

    # off-diagonal block with row lengths that differ between the operands:
    # |S(j)| of the Jaccard denominator is the length of row j of A_j
    h = g["offdiag_jaccard_pair"]
    Ai, Aj = _csr(h["Ai"], values=False), _csr(h["Aj"], values=False)
    for sr in ("count", "jaccard"):
        R = oracle.offdiag(Ai, Aj, sr, lib=lib)
        e = h["offdiag_" + sr]
        np.testing.assert_array_equal(R.row_ptr, e["row_ptr"])
        np.testing.assert_array_equal(R.col_idx, e["col_idx"])
        if sr == "count":
            np.testing.assert_array_equal(R.values, e["values"])
        else:
            want = np.float32(e["numerator"]) / np.float32(e["denominator"])
            np.testing.assert_array_equal(R.values.view(np.uint32), want.view(np.uint32))


def test_golden_hand_worked():
    check_golden()


# --------------------------------------------------------------------------
# dense brute force (numpy A @ A.T) on many tiny inputs


def brute_lower(A):
    D, P = dense_of(A)
    C = D @ D.T
    S = (P.astype(np.int64) @ P.T.astype(np.int64)) > 0
    return np.tril(C), np.tril(S)


def check_brute(seed_count=40, lib=None):
    rng = np.random.default_rng(12345)
    for t in range(seed_count):
        m = int(rng.integers(0, 40))
        n = int(rng.integers(1, 60))
        dens = float(rng.choice([0.02, 0.08, 0.2, 0.5]))
        A = random_csr(rng, m, n, dens, zeros=0.1)
        C, S = brute_lower(A)
        R = oracle.lower(A, "f64", lib=lib)
        assert_canonical_rows(R.row_ptr, R.col_idx)
        RD, RP = result_to_dense(R, m)
        np.testing.assert_array_equal(RP, S, err_msg=f"structure case {t}")
        np.testing.assert_allclose(RD, C, rtol=1e-12, atol=1e-12, err_msg=f"values case {t}")
        # count semiring: number of shared columns
        Dp, Pp = dense_of(A)
        cnt = np.tril(Pp.astype(np.int64) @ Pp.T.astype(np.int64))
        R = oracle.lower(A.with_values(None), "count", lib=lib)
        RD, RP = result_to_dense(R, m)
        np.testing.assert_array_equal(RP, S)
        np.testing.assert_array_equal(RD.astype(np.int64), cnt)
        # fp32: inputs rounded to fp32, products exact in fp64, one rounding at the end
        A32 = A.with_values(A.values.astype(np.float32))
        C32, _ = brute_lower(A32.with_values(A32.values.astype(np.float64)))
        R = oracle.lower(A32, "f32", lib=lib)
        RD, RP = result_to_dense(R, m)
        np.testing.assert_array_equal(RP, S)
        np.testing.assert_allclose(RD, C32.astype(np.float32), rtol=2e-7, atol=1e-30)
        # Jaccard from the count matrix and row lengths, in float32
        lens = np.diff(A.row_ptr)
        R = oracle.lower(A.with_values(None), "jaccard", lib=lib)
        rows = np.repeat(np.arange(m), np.diff(R.row_ptr))
        c = cnt[rows, R.col_idx]
        want = np.float32(c) / np.float32(lens[rows] + lens[R.col_idx] - c)
        np.testing.assert_array_equal(R.values.view(np.uint32), want.astype(np.float32).view(np.uint32))


def test_dense_brute_force():
    check_brute()


def check_offdiag_brute(lib=None):
    rng = np.random.default_rng(777)
    for t in range(30):
        mi, mj = int(rng.integers(0, 30)), int(rng.integers(0, 30))
        n = int(rng.integers(1, 50))
        # the two operands have different densities, so their row lengths differ
        Ai = random_csr(rng, mi, n, 0.15)
        Aj = random_csr(rng, mj, n, float(rng.choice([0.05, 0.3])))
        Di, Pi = dense_of(Ai)
        Dj, Pj = dense_of(Aj)
        R = oracle.offdiag(Ai, Aj, "f64", lib=lib)
        RD, RP = result_to_dense(R, mj)
        S = (Pi.astype(int) @ Pj.T.astype(int)) > 0
        np.testing.assert_array_equal(RP, S)
        np.testing.assert_allclose(RD, Di @ Dj.T, rtol=1e-12, atol=1e-12)
        # counts: the integer pattern product
        cnt = Pi.astype(np.int64) @ Pj.T.astype(np.int64)
        R = oracle.offdiag(Ai.with_values(None), Aj.with_values(None), "count", lib=lib)
        RD, RP = result_to_dense(R, mj)
        np.testing.assert_array_equal(RP, S)
        np.testing.assert_array_equal(RD.astype(np.int64), cnt)
        # Jaccard: c / (|S_i| + |S_j| - c) in float32, |S_i| a row length of
        # A_i and |S_j| one of A_j (the rows of the two operands differ)
        R = oracle.offdiag(Ai.with_values(None), Aj.with_values(None), "jaccard", lib=lib)
        rows = np.repeat(np.arange(mi), np.diff(R.row_ptr))
        c = cnt[rows, R.col_idx]
        li, lj = np.diff(Ai.row_ptr), np.diff(Aj.row_ptr)
        want = np.float32(c) / np.float32(li[rows] + lj[R.col_idx] - c)
        np.testing.assert_array_equal(R.col_idx, np.nonzero(S)[1])
        np.testing.assert_array_equal(R.values.view(np.uint32), want.astype(np.float32).view(np.uint32))
        # fp32: inputs rounded to float32, one rounding of the exact sum
        Ai32 = Ai.with_values(Ai.values.astype(np.float32))
        Aj32 = Aj.with_values(Aj.values.astype(np.float32))
        D32 = dense_of(Ai32.with_values(Ai32.values.astype(np.float64)))[0] @ \
            dense_of(Aj32.with_values(Aj32.values.astype(np.float64)))[0].T
        R = oracle.offdiag(Ai32, Aj32, "f32", lib=lib)
        RD, RP = result_to_dense(R, mj)
        np.testing.assert_array_equal(RP, S)
        np.testing.assert_allclose(RD, D32.astype(np.float32), rtol=2e-7, atol=1e-30)


def test_offdiag_brute_force():
    check_offdiag_brute()


def test_threads_give_the_same_result():
    # the row-sharded driver runs the same per-row code: identical output,
    # bit for bit, for every semiring, a row subset and the off-diagonal call
    rng = np.random.default_rng(9)
    A = random_csr(rng, 20000 // 100, 300, 0.03)
    B = random_csr(rng, 150, 300, 0.03)
    big = W.make("kmer_i32", 1, 6)["A"]
    for Ain, sr in ((A, "f64"), (A.with_values(A.values.astype(np.float32)), "f32"),
                    (big, "count"), (big, "jaccard")):
        one = oracle.lower(Ain, sr)
        many = oracle.lower(Ain, sr, threads=4)
        for f in ("row_ptr", "col_idx", "sum_abs", "count"):
            np.testing.assert_array_equal(getattr(one, f), getattr(many, f))
        np.testing.assert_array_equal(one.values.view(np.uint8), many.values.view(np.uint8))
    rows = np.array([17, 3, 3, 150, 0])
    np.testing.assert_array_equal(oracle.lower(A, "f64", rows=rows).col_idx,
                                  oracle.lower(A, "f64", rows=rows, threads=3).col_idx)
    one, many = oracle.offdiag(A, B, "f64"), oracle.offdiag(A, B, "f64", threads=5)
    np.testing.assert_array_equal(one.row_ptr, many.row_ptr)
    np.testing.assert_array_equal(one.values, many.values)


def test_row_subset_matches_full():
    rng = np.random.default_rng(3)
    A = random_csr(rng, 50, 40, 0.1)
    full = oracle.lower(A, "f64")
    rows = np.array([49, 0, 17, 17, 3])
    sub = oracle.lower(A, "f64", rows=rows)
    for q, i in enumerate(rows):
        a, b = full.row_ptr[i], full.row_ptr[i + 1]
        c, d = sub.row_ptr[q], sub.row_ptr[q + 1]
        np.testing.assert_array_equal(full.col_idx[a:b], sub.col_idx[c:d])
        np.testing.assert_array_equal(full.values[a:b], sub.values[c:d])


# --------------------------------------------------------------------------
# scipy.sparse on the tiny workload and on scaled-down versions of the others


def _scipy_lower(A):
    S = to_scipy(A)
    C = sp.tril(S @ S.T).tocsr()
    Pt = to_scipy(A, np.ones(len(A.col_idx)))
    St = sp.tril(Pt @ Pt.T).tocsr()
    St.sort_indices()
    C.sort_indices()
    return C, St


@pytest.mark.parametrize("name,shift", [("tiny_uniform_f64", 0), ("kmer_i32", 6), ("rmat20_f32", 9),
                                        ("offdiag_f64", 6), ("jaccard_large", 9)])
def test_scipy_on_workloads(name, shift):
    w = W.make(name, 1, shift)
    A = w["A"]
    sr = w["semiring"]
    R = oracle.lower(A, sr)
    _, St = _scipy_lower(A)
    # structure from the pattern product (no cancellation possible with all-ones)
    np.testing.assert_array_equal(R.row_ptr, St.indptr)
    np.testing.assert_array_equal(R.col_idx, St.indices)
    if sr == "count":
        np.testing.assert_array_equal(R.values, St.data.astype(np.int32))
    elif sr == "f64":
        C, _ = _scipy_lower(A)
        Cd = C.toarray() if C.shape[0] <= 4096 else None
        vals = np.asarray(C[np.repeat(np.arange(A.nrows), np.diff(R.row_ptr)), R.col_idx]).ravel() \
            if Cd is None else Cd[np.repeat(np.arange(A.nrows), np.diff(R.row_ptr)), R.col_idx]
        np.testing.assert_allclose(R.values, vals, rtol=1e-12)
    elif sr == "f32":
        A64 = A.with_values(A.values.astype(np.float64))
        S = to_scipy(A64)
        C = sp.tril(S @ S.T).tocsr()
        C.sort_indices()
        np.testing.assert_array_equal(C.indices, R.col_idx)
        np.testing.assert_allclose(R.values, C.data.astype(np.float32), rtol=1e-6)
    if "offdiag" in w["ops"]:
        Ai, Aj = w["A"], w["B"]
        R = oracle.offdiag(Ai, Aj, "f64")
        C = (to_scipy(Ai) @ to_scipy(Aj).T).tocsr()
        C.sort_indices()
        Pc = (to_scipy(Ai, np.ones(Ai.nnz)) @ to_scipy(Aj, np.ones(Aj.nnz)).T).tocsr()
        Pc.sort_indices()
        np.testing.assert_array_equal(R.row_ptr, Pc.indptr)
        np.testing.assert_array_equal(R.col_idx, Pc.indices)
        np.testing.assert_allclose(R.values, C.data, rtol=1e-12)


# --------------------------------------------------------------------------
# invariants and closed forms


def _FL(A):
    c = np.bincount(A.col_idx, minlength=A.ncols).astype(np.int64)
    return int((c * (c + 1) // 2).sum())


def check_invariants(A, lib=None):
    m = A.nrows
    R = oracle.lower(A.with_values(None), "count", lib=lib)
    # half-work identity: total lower multiply-adds = sum_k c_k (c_k + 1) / 2 = (F + nnz) / 2
    c = np.bincount(A.col_idx, minlength=A.ncols).astype(np.int64)
    assert int(R.values.astype(np.int64).sum()) == _FL(A) == (int((c * c).sum()) + A.nnz) // 2
    # every entry of the lower part
    rows = np.repeat(np.arange(m), np.diff(R.row_ptr))
    assert np.all(R.col_idx <= rows)
    # diagonal: the last entry of each non-empty row, equal to the row's squared norm
    Rf = oracle.lower(A, "f64", lib=lib)
    lens = np.diff(A.row_ptr)
    ne = np.flatnonzero(lens > 0)
    last = Rf.row_ptr[ne + 1] - 1
    np.testing.assert_array_equal(Rf.col_idx[last], ne)
    sq = np.add.reduceat(A.values ** 2, A.row_ptr[ne]) if len(ne) else np.zeros(0)
    np.testing.assert_allclose(Rf.values[last], sq, rtol=1e-12)
    assert np.all(np.diff(Rf.row_ptr)[lens == 0] == 0)
    # mirror: exact symmetry and the entry count 2 nnz(C_L) - #non-empty rows
    M = oracle.mirror(m, Rf.row_ptr, Rf.col_idx, Rf.values, lib=lib)
    assert M.nnz == 2 * Rf.nnz - len(ne)
    Ms = sp.csr_matrix((M.values, M.col_idx, M.row_ptr), shape=(m, m))
    assert (Ms != Ms.T).nnz == 0
    assert_canonical_rows(M.row_ptr, M.col_idx)
    # global checksum: 2 sum_{j<i} C_L + sum_i C_L(i,i) = sum_k (sum_i A(i,k))^2
    colsum = np.bincount(A.col_idx, weights=A.values, minlength=A.ncols)
    diag_sum = Rf.values[last].sum()
    total = 2.0 * Rf.values.sum() - diag_sum
    np.testing.assert_allclose(total, (colsum ** 2).sum(), rtol=1e-10)
    # offdiag(A, A) is the full product: equal to the mirror
    O = oracle.offdiag(A, A, "f64", lib=lib)
    np.testing.assert_array_equal(O.row_ptr, M.row_ptr)
    np.testing.assert_array_equal(O.col_idx, M.col_idx)
    np.testing.assert_allclose(O.values, M.values, rtol=1e-12)


def test_invariants_random():
    rng = np.random.default_rng(99)
    for _ in range(10):
        A = random_csr(rng, int(rng.integers(1, 80)), int(rng.integers(1, 80)), 0.08, signed=False)
        check_invariants(A)


def test_invariants_workloads():
    for name, shift in [("kmer_i32", 7), ("rmat20_f32", 10), ("jaccard_large", 10), ("tiny_uniform_f64", 2)]:
        A = W.make(name, 1, shift)["A"]
        vals = A.values if A.values is not None else np.ones(A.nnz)
        check_invariants(A.with_values(vals.astype(np.float64)))


def test_offdiag_transpose_identity():
    # C_ij = C_ji^T (Sec. III-A): offdiag(Ai, Aj) is the transpose of offdiag(Aj, Ai)
    rng = np.random.default_rng(5)
    Ai = random_csr(rng, 37, 50, 0.1)
    Aj = random_csr(rng, 23, 50, 0.1)
    X = oracle.offdiag(Ai, Aj, "f64")
    Y = oracle.offdiag(Aj, Ai, "f64")
    Xs = sp.csr_matrix((X.values, X.col_idx, X.row_ptr), shape=(37, 23))
    Yt = sp.csr_matrix((Y.values, Y.col_idx, Y.row_ptr), shape=(23, 37)).T.tocsr()
    Yt.sort_indices()
    np.testing.assert_array_equal(Xs.indptr, Yt.indptr)
    np.testing.assert_array_equal(Xs.indices, Yt.indices)
    np.testing.assert_allclose(Xs.data, Yt.data, rtol=1e-12)


def _transpose_result(R, ncols):
    S = sp.csr_matrix((R.values, R.col_idx, R.row_ptr), shape=(R.nrows, ncols)).T.tocsr()
    S.sort_indices()
    return S


def test_offdiag_halves_cover_the_pair():
    # Sec. III-A / Algorithm 3: the lower process of a pair computes the top
    # rows of C_ij, its partner the right columns of C_ji; row r of C_ij is
    # column r of C_ji, so the two halves are disjoint and hold all of C_ij
    rng = np.random.default_rng(12)
    for mi, mj in ((37, 23), (1, 5), (2, 1), (40, 40), (0, 3)):
        Ai = random_csr(rng, mi, 30, 0.12)
        Aj = random_csr(rng, mj, 30, 0.12)
        full = oracle.offdiag(Ai, Aj, "f64")
        top = oracle.offdiag_half(Ai, Aj, "top", "f64")
        right = oracle.offdiag_half(Aj, Ai, "right", "f64")  # part of C_ji, m_j x m_i
        assert top.nrows == mi // 2 and right.nrows == mj
        assert np.all(right.col_idx >= mi // 2)
        # the top rows are the full block's first rows, unchanged
        cut = full.row_ptr[mi // 2]
        np.testing.assert_array_equal(top.row_ptr, full.row_ptr[:mi // 2 + 1])
        np.testing.assert_array_equal(top.col_idx, full.col_idx[:cut])
        np.testing.assert_array_equal(top.values, full.values[:cut])
        # the right half of C_ji, transposed, is the rest of C_ij (same products
        # in the same order of k, so bit for bit)
        rt = _transpose_result(right, mi)   # m_i x m_j, rows < m_i // 2 empty
        assert rt.indptr[mi // 2] == 0
        np.testing.assert_array_equal(rt.indptr[mi // 2:] , full.row_ptr[mi // 2:] - cut)
        np.testing.assert_array_equal(rt.indices, full.col_idx[cut:])
        np.testing.assert_array_equal(rt.data, full.values[cut:])


def test_offdiag_half_brute_force():
    rng = np.random.default_rng(13)
    for t in range(20):
        mi, mj, n = int(rng.integers(0, 20)), int(rng.integers(0, 20)), int(rng.integers(1, 30))
        Ai = random_csr(rng, mi, n, 0.2)
        Aj = random_csr(rng, mj, n, 0.2)
        Di, Pi = dense_of(Ai)
        Dj, Pj = dense_of(Aj)
        P = (Pi.astype(int) @ Pj.T.astype(int)) > 0
        D = Di @ Dj.T
        top = oracle.offdiag_half(Ai, Aj, "top", "f64")
        TD, TP = result_to_dense(top, mj)
        np.testing.assert_array_equal(TP, P[:mi // 2])
        np.testing.assert_allclose(TD, D[:mi // 2], rtol=1e-12, atol=1e-12)
        right = oracle.offdiag_half(Ai, Aj, "right", "f64")
        RD, RP = result_to_dense(right, mj)
        want = P.copy()
        want[:, :mj // 2] = False
        np.testing.assert_array_equal(RP, want)
        np.testing.assert_allclose(RD, np.where(want, D, 0.0), rtol=1e-12, atol=1e-12)


def test_symm_is_A_times_AT_x():
    # Eq. (spmv) on C_L = tril(A A^T): C X = A (A^T X), the route that never
    # forms C (Sec. V-F), a different summation entirely
    rng = np.random.default_rng(21)
    for m, n, k in ((40, 30, 1), (25, 60, 3), (1, 5, 2), (30, 1, 4)):
        A = random_csr(rng, m, n, 0.15)
        D, _ = dense_of(A)
        X = rng.standard_normal((m, k))
        L = oracle.lower(A, "f64")
        Y, S = oracle.symm(m, L.row_ptr, L.col_idx, L.values, X)
        want = D @ (D.T @ X)
        np.testing.assert_allclose(Y, want, rtol=0, atol=1e-12 * max(1.0, float(np.abs(D).sum() ** 2)))
        assert np.all(S >= np.abs(Y) - 1e-12)


def test_symm_matches_mirrored_matrix():
    # against the materialised full matrix (the mirror) times X, and unit
    # vectors pick out columns of C
    rng = np.random.default_rng(22)
    m = 35
    A = random_csr(rng, m, 50, 0.1)
    L = oracle.lower(A, "f64")
    M = oracle.mirror(m, L.row_ptr, L.col_idx, L.values)
    C = sp.csr_matrix((M.values, M.col_idx, M.row_ptr), shape=(m, m)).toarray()
    X = rng.standard_normal((m, 5))
    Y, _ = oracle.symm(m, L.row_ptr, L.col_idx, L.values, X)
    np.testing.assert_allclose(Y, C @ X, rtol=1e-12, atol=1e-12)
    E, _ = oracle.symm(m, L.row_ptr, L.col_idx, L.values, np.eye(m))
    np.testing.assert_array_equal(E, C)
    # an empty lower part gives zeros
    Z, _ = oracle.symm(3, np.zeros(4, np.int64), np.zeros(0, np.int32), np.zeros(0), np.ones((3, 2)))
    np.testing.assert_array_equal(Z, 0.0)


def _hcat(A1, A2):
    D1, P1 = dense_of(A1)
    D2, P2 = dense_of(A2)
    return csr_from_dense(np.hstack([D1, D2]), pattern=np.hstack([P1, P2]))


def test_accumulate_is_concatenation():
    # one stage at a time: lower(A1) + tril(A2 A2^T) = lower([A1 A2]) (Sec. III-A)
    rng = np.random.default_rng(31)
    for m in (30, 1, 17):
        A1 = random_csr(rng, m, 20, 0.15)
        A2 = random_csr(rng, m, 25, 0.15)
        A3 = random_csr(rng, m, 9, 0.3)
        for sr in ("f64", "count"):
            acc = oracle.lower(A1 if sr == "f64" else A1.with_values(None), sr)
            for Ak in (A2, A3):
                acc = oracle.lower_accumulate(acc, Ak if sr == "f64" else Ak.with_values(None), sr)
            A = _hcat(_hcat(A1, A2), A3)
            ref = oracle.lower(A if sr == "f64" else A.with_values(None), sr)
            np.testing.assert_array_equal(acc.row_ptr, ref.row_ptr)
            np.testing.assert_array_equal(acc.col_idx, ref.col_idx)
            if sr == "count":
                np.testing.assert_array_equal(acc.values, ref.values)
            else:
                np.testing.assert_allclose(acc.values, ref.values, rtol=1e-12, atol=1e-12)


def test_accumulate_f32_is_one_float_addition():
    # F32 stages (Sec. III-A, C_ii = sum_s SYRK(A_is)): each stage is rounded to
    # float32 once, and an entry present in both parts is one correctly rounded
    # float32 addition of the two float32 values (numpy float32 arithmetic);
    # an entry in one part keeps its value.  Against the one-shot lower part of
    # the concatenation the result stays within the fp32 bar.
    rng = np.random.default_rng(33)
    for m in (30, 1, 17):
        A1 = random_csr(rng, m, 20, 0.2, dtype=np.float32, signed=False)
        A2 = random_csr(rng, m, 25, 0.2, dtype=np.float32, signed=False)
        P = oracle.lower(A1, "f32")
        T = oracle.lower(A2, "f32")
        acc = oracle.lower_accumulate(P, A2, "f32")
        want = {}
        for R in (P, T):
            rows = np.repeat(np.arange(m), np.diff(R.row_ptr))
            for i, j, v in zip(rows, R.col_idx, R.values):
                key = (int(i), int(j))
                want[key] = np.float32(want[key] + v) if key in want else np.float32(v)
        keys = sorted(want)
        rp = np.zeros(m + 1, dtype=np.int64)
        np.cumsum(np.bincount([k[0] for k in keys], minlength=m), out=rp[1:])
        np.testing.assert_array_equal(acc.row_ptr, rp)
        np.testing.assert_array_equal(acc.col_idx, [k[1] for k in keys])
        got = np.asarray(acc.values, dtype=np.float32)
        np.testing.assert_array_equal(got.view(np.uint32),
                                      np.array([want[k] for k in keys], dtype=np.float32).view(np.uint32))
        ref = oracle.lower(_hcat(A1, A2).with_values(None), "count")
        np.testing.assert_array_equal(acc.col_idx, ref.col_idx)
        A = _hcat(A1, A2)
        one = oracle.lower(A.with_values(A.values.astype(np.float32)), "f32")
        np.testing.assert_allclose(got, one.values, rtol=1e-5, atol=0)


def test_accumulate_from_empty():
    rng = np.random.default_rng(32)
    A = random_csr(rng, 25, 30, 0.12)
    empty = oracle.Result(25, 25, np.zeros(26, np.int64), np.zeros(0, np.int32), np.zeros(0))
    acc = oracle.lower_accumulate(empty, A, "f64")
    ref = oracle.lower(A, "f64")
    np.testing.assert_array_equal(acc.row_ptr, ref.row_ptr)
    np.testing.assert_array_equal(acc.col_idx, ref.col_idx)
    np.testing.assert_array_equal(acc.values, ref.values)


def test_concatenation_sums_stages():
    # C_ii = sum_s SYRK(A_is) (Sec. III-A): lower([A1 A2]) = lower(A1) + lower(A2)
    rng = np.random.default_rng(8)
    D1, P1 = dense_of(random_csr(rng, 30, 20, 0.15))
    D2, P2 = dense_of(random_csr(rng, 30, 25, 0.15))
    A = csr_from_dense(np.hstack([D1, D2]), pattern=np.hstack([P1, P2]))
    A1 = csr_from_dense(D1, pattern=P1)
    A2 = csr_from_dense(D2, pattern=P2)
    R = oracle.lower(A, "f64")
    R1 = oracle.lower(A1, "f64")
    R2 = oracle.lower(A2, "f64")
    S = sp.csr_matrix((R.values, R.col_idx, R.row_ptr), shape=(30, 30))
    S12 = sp.csr_matrix((R1.values, R1.col_idx, R1.row_ptr), shape=(30, 30)) + \
        sp.csr_matrix((R2.values, R2.col_idx, R2.row_ptr), shape=(30, 30))
    np.testing.assert_allclose(S.toarray(), S12.toarray(), rtol=1e-12, atol=1e-14)


def test_special_cases():
    # identity -> identity
    m = 17
    I = csr_from_dense(np.eye(m))
    R = oracle.lower(I, "f64")
    np.testing.assert_array_equal(R.row_ptr, np.arange(m + 1))
    np.testing.assert_array_equal(R.col_idx, np.arange(m))
    np.testing.assert_array_equal(R.values, np.ones(m))
    # one all-ones column -> dense lower triangle of ones, m (m + 1) / 2 entries
    D = np.zeros((m, 3))
    D[:, 1] = 1.0
    R = oracle.lower(csr_from_dense(D), "count")
    assert R.nnz == m * (m + 1) // 2
    assert np.all(R.values == 1)
    # disjoint supports -> diagonal only
    D = np.zeros((m, 2 * m))
    D[np.arange(m), 2 * np.arange(m)] = 2.0
    D[np.arange(m), 2 * np.arange(m) + 1] = 3.0
    R = oracle.lower(csr_from_dense(D), "f64")
    np.testing.assert_array_equal(R.col_idx, np.arange(m))
    np.testing.assert_array_equal(R.values, np.full(m, 13.0))
    # A = [B; B] -> C_L = [[tril(BB^T), 0], [BB^T, tril(BB^T)]]
    rng = np.random.default_rng(11)
    Bd, Bp = dense_of(random_csr(rng, 9, 12, 0.3))
    A = csr_from_dense(np.vstack([Bd, Bd]), pattern=np.vstack([Bp, Bp]))
    R = oracle.lower(A, "f64")
    RD, RP = result_to_dense(R, 18)
    G = Bd @ Bd.T
    np.testing.assert_allclose(RD[9:, :9], G, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(RD[:9, :9], np.tril(G), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(RD[9:, 9:], np.tril(G), rtol=1e-12, atol=1e-14)
    # empty matrix and empty rows
    E = CSR(5, 4, np.zeros(6, dtype=np.int64), np.zeros(0, dtype=np.int32), np.zeros(0))
    R = oracle.lower(E, "f64")
    assert R.nnz == 0 and np.all(R.row_ptr == 0)
    E0 = CSR(0, 4, np.zeros(1, dtype=np.int64), np.zeros(0, dtype=np.int32), np.zeros(0))
    assert oracle.lower(E0, "f64").nnz == 0


def test_permutations():
    rng = np.random.default_rng(21)
    A = random_csr(rng, 40, 60, 0.08, signed=False)
    D, P = dense_of(A)
    R = oracle.lower(A, "f64")
    M = oracle.mirror(40, R.row_ptr, R.col_idx, R.values)
    C = sp.csr_matrix((M.values, M.col_idx, M.row_ptr), shape=(40, 40)).toarray()
    # column permutation leaves C unchanged
    q = rng.permutation(60)
    Rq = oracle.lower(csr_from_dense(D[:, q], pattern=P[:, q]), "f64")
    np.testing.assert_array_equal(Rq.col_idx, R.col_idx)
    np.testing.assert_allclose(Rq.values, R.values, rtol=1e-12)
    # row permutation p gives C[p][:, p]
    p = rng.permutation(40)
    Rp = oracle.lower(csr_from_dense(D[p], pattern=P[p]), "f64")
    Mp = oracle.mirror(40, Rp.row_ptr, Rp.col_idx, Rp.values)
    Cp = sp.csr_matrix((Mp.values, Mp.col_idx, Mp.row_ptr), shape=(40, 40)).toarray()
    np.testing.assert_allclose(Cp, C[np.ix_(p, p)], rtol=1e-12, atol=1e-15)


def test_rejects_non_canonical():
    A = CSR(2, 4, np.array([0, 2, 3]), np.array([2, 1, 0], dtype=np.int32), np.ones(3))
    with pytest.raises(oracle.OracleError):
        oracle.lower(A, "f64")
    A = CSR(2, 4, np.array([0, 2, 3]), np.array([1, 1, 0], dtype=np.int32), np.ones(3))
    with pytest.raises(oracle.OracleError):
        oracle.lower(A, "f64")
    A = CSR(2, 4, np.array([0, 2, 3]), np.array([1, 4, 0], dtype=np.int32), np.ones(3))
    with pytest.raises(oracle.OracleError):
        oracle.lower(A, "f64")
    with pytest.raises(oracle.OracleError):  # entry above the diagonal
        oracle.mirror(2, np.array([0, 2, 3]), np.array([0, 1, 0], dtype=np.int32), np.ones(3))


# --------------------------------------------------------------------------
# planted mistakes: each mutant of the oracle source must fail a pin

MUTANTS = {
    "prune_drops_diagonal": ("if (lower && j > i) break;", "if (lower && j >= i) break;"),
    "no_prune": ("if (lower && j > i) break;", "if (false && j > i) break;"),
    "sum_instead_of_product": ("const double prod = a * T.val[p];", "const double prod = a + T.val[p];"),
    "self_value_squared": ("const double prod = a * T.val[p];", "const double prod = a * a;"),
    "transpose_row_off_by_one": ("T.row[slot] = static_cast<int32_t>(r);",
                                 "T.row[slot] = static_cast<int32_t>(r > 0 ? r - 1 : r);"),
    "jaccard_plus_c": ("len_i + len_j - static_cast<int64_t>(a.count)", "len_i + len_j + static_cast<int64_t>(a.count)"),
    "jaccard_len_i_twice": ("const int64_t len_j = B.rp[j + 1] - B.rp[j];", "const int64_t len_j = len_i;"),
    "mirror_skips_transposed": ("if (ci[e] < r) full[ci[e]].push_back", "if (ci[e] < r - 1) full[ci[e]].push_back"),
    "count_double": ("s.count += 1u;", "s.count += 2u;"),
    # off the diagonal, |S(j)| taken from the left operand A_i instead of A_j
    # (kept in range: only where A_i has at least as many rows)
    "jaccard_len_j_from_left": ("emit_row(R, acc, sr, A.rp[i + 1] - A.rp[i], B);",
                                "emit_row(R, acc, sr, A.rp[i + 1] - A.rp[i], (lower || A.m < B.m) ? B : A);"),
}


def _all_pins(lib):
    check_golden(lib)
    check_brute(12, lib)
    check_offdiag_brute(lib)
    rng = np.random.default_rng(4)
    for _ in range(3):
        check_invariants(random_csr(rng, 30, 25, 0.12, signed=False), lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_fail(name, tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    src = open(os.path.join(os.path.dirname(oracle.__file__), "spsyrk_oracle.cpp")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    path = tmp_path / "mutant.cpp"
    path.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", "-pthread", "-o", str(so), str(path)])
    lib = oracle._load(str(so))
    with pytest.raises((AssertionError, oracle.OracleError)):
        _all_pins(lib)


def test_unmutated_passes_all_pins():
    _all_pins(oracle._load())
