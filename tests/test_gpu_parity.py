"""GPU parity: the HIP library through its C-ABI against the CPU oracle.

Inputs are seeded and synthetic: hand-worked fixtures, random matrices with
empty rows, stored zeros and negative values, the degenerate shapes, rows
that overflow the light path (long rows, rows with many products), and the
five workloads at reduced size (several tiles and a ragged tail each).
"""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2608_09713_amd as sp
from paper_2608_09713_amd import workloads as W
from paper_2608_09713_amd.workloads import CSR
from tests.helpers import csr_from_dense, random_csr
from tests.parity import compare_full

pytestmark = pytest.mark.gpu

SEMIRINGS = ["f64", "f32", "count", "jaccard"]
VDT = {"f64": np.float64, "f32": np.float32, "count": None, "jaccard": None}


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available()
    sp.library()
    return "cuda:0"


def upload(A, semiring, dev):
    vals = None
    if VDT[semiring] is not None:
        vals = (A.values if A.values is not None else np.ones(A.nnz)).astype(VDT[semiring])
    return sp.DeviceCSR.from_host(A.with_values(vals), dev)


def run_lower(A, semiring, dev, what):
    print(f"[lower {semiring}] {what} m={A.nrows} n={A.ncols} nnz={A.nnz}", flush=True)
    C = sp.lower(upload(A, semiring, dev), semiring)
    ref = oracle.lower(A.with_values(None if VDT[semiring] is None else A.values.astype(VDT[semiring])), semiring)
    compare_full(C, ref, semiring, what)
    return C


def test_golden_on_gpu(dev):
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_small.json")))
    P = CSR(4, 5, np.array(g["P"]["row_ptr"]), np.array(g["P"]["col_idx"], dtype=np.int32),
            np.array(g["P"]["values"]))
    C = sp.lower(upload(P, "f64", dev), "f64")
    rp, ci, v = C.to_host()
    e = g["P"]["lower_f64"]
    np.testing.assert_array_equal(rp, e["row_ptr"])
    np.testing.assert_array_equal(ci, e["col_idx"])
    np.testing.assert_array_equal(v, e["values"])
    M = sp.mirror(C, "f64")
    rp, ci, v = M.to_host()
    e = g["P"]["mirror_f64"]
    np.testing.assert_array_equal(rp, e["row_ptr"])
    np.testing.assert_array_equal(ci, e["col_idx"])
    np.testing.assert_array_equal(v, e["values"])
    C = sp.lower(upload(P, "jaccard", dev), "jaccard")
    e = g["P"]["lower_jaccard"]
    want = (np.float32(e["numerator"]) / np.float32(e["denominator"])).view(np.uint32)
    np.testing.assert_array_equal(C.to_host()[2].view(np.uint32), want)
    # off-diagonal block whose operands' rows differ in length
    h = g["offdiag_jaccard_pair"]
    Ai, Aj = (CSR(h[k]["nrows"], h[k]["ncols"], np.array(h[k]["row_ptr"]), np.array(h[k]["col_idx"], dtype=np.int32),
                  None) for k in ("Ai", "Aj"))
    for sr in ("count", "jaccard"):
        C = sp.offdiag(upload(Ai, sr, dev), upload(Aj, sr, dev), sr)
        rp, ci, v = C.to_host()
        e = h["offdiag_" + sr]
        np.testing.assert_array_equal(rp, e["row_ptr"])
        np.testing.assert_array_equal(ci, e["col_idx"])
        if sr == "count":
            np.testing.assert_array_equal(v, e["values"])
        else:
            want = (np.float32(e["numerator"]) / np.float32(e["denominator"])).view(np.uint32)
            np.testing.assert_array_equal(v.view(np.uint32), want)


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_random_small(dev, semiring):
    rng = np.random.default_rng(2024)
    for t in range(12):
        m = int(rng.integers(1, 300))
        n = int(rng.integers(1, 400))
        A = random_csr(rng, m, n, float(rng.choice([0.005, 0.03, 0.1])), zeros=0.05)
        run_lower(A, semiring, dev, f"random case {t}")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_degenerate_shapes(dev, semiring):
    cases = {
        "empty_matrix": CSR(7, 5, np.zeros(8, np.int64), np.zeros(0, np.int32), np.zeros(0)),
        "one_row": csr_from_dense(np.array([[1.0, 0.0, 2.0]])),
        "one_column": csr_from_dense(np.ones((9, 1))),
        "identity": csr_from_dense(np.eye(33)),
        "empty_rows_between": csr_from_dense(np.array([[0, 0, 0], [1.0, 2.0, 0], [0, 0, 0], [3.0, 0, 4.0],
                                                       [0, 0, 0]])),
    }
    for name, A in cases.items():
        run_lower(A, semiring, dev, name)
    E0 = CSR(0, 3, np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0))
    C = sp.lower(upload(E0, semiring, dev), semiring)
    assert C.nnz == 0 and C.row_ptr.numel() == 1


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_dense_column_uses_heavy_rows(dev, semiring):
    # one all-ones column over 2500 rows: row i has i products, so rows past
    # the light limit go to the dense-tile path; output is the full lower triangle
    m = 2500
    D = np.zeros((m, 4))
    D[:, 2] = 1.0
    D[::3, 0] = 0.5
    A = csr_from_dense(D)
    run_lower(A, semiring, dev, "dense column")
    assert sp.stats()["heavy_rows"] > 0


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_long_rows_use_heavy_rows(dev, semiring):
    rng = np.random.default_rng(7)
    m, n = 300, 5000
    D = np.zeros((m, n))
    P = rng.random((m, n)) < 0.01
    P[5, :1200] = True          # more entries than the light path takes
    P[200, ::3] = True
    D[P] = rng.random(P.sum()) + 0.5
    A = csr_from_dense(D, pattern=P)
    run_lower(A, semiring, dev, "long rows")
    assert sp.stats()["heavy_rows"] >= 2


def _hub_csr(rng, m, n, per_row, hub_rows, dtype=np.float64):
    # per_row random columns in [2, n) per row; columns 0 and 1 are hubs held
    # by hub_rows random rows each, so these rows meet thousands of partners
    # spread over the whole row range
    c = rng.integers(2, n, size=(m, per_row + 2))
    c[:, :2] = -1
    for k in range(2):
        c[rng.choice(m, size=hub_rows, replace=False), k] = k
    c.sort(axis=1)
    keep = c >= 0
    keep[:, 1:] &= c[:, 1:] != c[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(keep.sum(axis=1))
    ci = c[keep].astype(np.int32)
    return CSR(m, n, rp, ci, (rng.random(len(ci)) + 0.5).astype(dtype))


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_heavy_rows_across_windows(dev, semiring):
    # heavy rows whose partners spread over 300000 rows: the numeric pass
    # sweeps three windows of 2^17 columns (the last one partial), the
    # symbolic pass two of 2^18; lower and off-diagonal products
    rng = np.random.default_rng(57)
    A = _hub_csr(rng, 300000, 1 << 20, 3, 3000)
    run_lower(A, semiring, dev, "heavy rows across windows")
    assert sp.stats()["heavy_rows"] > 1000
    vdt = VDT[semiring]
    Ai = _hub_csr(rng, 270000, 1 << 20, 3, 2000)
    Aj = _hub_csr(rng, 280000, 1 << 20, 3, 2000)
    O = sp.offdiag(upload(Ai, semiring, dev), upload(Aj, semiring, dev), semiring)
    assert sp.stats()["heavy_rows"] > 1000
    ref = oracle.offdiag(Ai.with_values(None if vdt is None else Ai.values.astype(vdt)),
                         Aj.with_values(None if vdt is None else Aj.values.astype(vdt)), semiring)
    compare_full(O, ref, semiring, "heavy offdiag across windows")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_light_rows_with_many_shared_columns(dev, semiring):
    # few columns, so that pairs of rows share several of them: the light
    # rows' buckets hold repeated columns (merges of 2..8 terms and larger)
    rng = np.random.default_rng(11)
    m, n, d = 300, 24, 8
    D = np.zeros((m, n))
    for i in range(m):
        D[i, rng.choice(n, size=d, replace=False)] = rng.random(d) + 0.25
    run_lower(csr_from_dense(D), semiring, dev, "shared columns")
    assert sp.stats()["light_rows"] > 0
    # identical rows: every output of a light row sums 10 terms of one column
    # index, more than a register-sorted bucket holds
    E = np.zeros((60, 50))
    E[:, 5:15] = rng.random((60, 10)) + 0.25
    run_lower(csr_from_dense(E), semiring, dev, "identical rows")
    assert sp.stats()["light_rows"] > 0


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_two_pass_path(dev, semiring, monkeypatch):
    # the two-pass kernels (directory lookups, symbolic then numeric) that the
    # off-diagonal call takes when the right operand has too many columns for
    # dense column starts; forced here on small inputs, light and heavy rows
    monkeypatch.setenv("SPSYRK_TWO_PASS", "1")
    rng = np.random.default_rng(99)
    A = random_csr(rng, 250, 300, 0.05, zeros=0.05)
    run_lower(A, semiring, dev, "two-pass lower")
    m = 2500
    D = np.zeros((m, 4))
    D[:, 2] = 1.0
    D[::3, 0] = 0.5
    run_lower(csr_from_dense(D), semiring, dev, "two-pass heavy rows")
    assert sp.stats()["heavy_rows"] > 0
    Ai = random_csr(rng, 120, 200, 0.05, signed=True)
    Aj = random_csr(rng, 90, 200, 0.05, signed=True)
    vdt = VDT[semiring]
    O = sp.offdiag(upload(Ai, semiring, dev), upload(Aj, semiring, dev), semiring)
    ref = oracle.offdiag(Ai.with_values(None if vdt is None else Ai.values.astype(vdt)),
                         Aj.with_values(None if vdt is None else Aj.values.astype(vdt)), semiring)
    compare_full(O, ref, semiring, "two-pass offdiag")


def test_many_chunks_full_parity(dev):
    # 2^21 rows: enough chunks per wavefront that the light-row kernel takes
    # runs of chunks from its counter; every row is compared with the oracle
    rng = np.random.default_rng(2024)
    m, n, per_row = 1 << 21, 1 << 22, 4
    c = np.sort(rng.integers(0, n, size=(m, per_row)), axis=1)
    keep = np.ones_like(c, dtype=bool)
    keep[:, 1:] = c[:, 1:] != c[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(keep.sum(axis=1))
    A = CSR(m, n, rp, c[keep].astype(np.int32), None)
    run_lower(A, "count", dev, "2^21 rows, 4 columns each")


def _rows_csr(rng, m, n, per_row, dtype=np.float64):
    c = np.sort(rng.integers(0, n, size=(m, per_row)), axis=1)
    keep = np.ones_like(c, dtype=bool)
    keep[:, 1:] = c[:, 1:] != c[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(keep.sum(axis=1))
    ci = c[keep].astype(np.int32)
    return CSR(m, n, rp, ci, rng.random(len(ci)).astype(dtype) + 0.5)


@pytest.mark.parametrize("semiring", ["f64", "count", "jaccard"])
def test_local_sort_path(dev, semiring, monkeypatch):
    # the column sort's local pass (high bits by passes, low bits inside
    # groups), forced on small inputs: 2^20 columns give 256 groups sorted in
    # LDS; 8192 columns give two groups of about 6000 entries, sorted over
    # global memory
    monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
    rng = np.random.default_rng(31)
    for m, n, per in ((3000, 1 << 20, 6), (3000, 8192, 4)):
        A = _rows_csr(rng, m, n, per)
        run_lower(A, semiring, dev, f"local sort m={m} n={n}")
        B = _rows_csr(rng, 2000, n, per)
        vdt = VDT[semiring]
        O = sp.offdiag(upload(A, semiring, dev), upload(B, semiring, dev), semiring)
        ref = oracle.offdiag(A.with_values(None if vdt is None else A.values.astype(vdt)),
                             B.with_values(None if vdt is None else B.values.astype(vdt)), semiring)
        compare_full(O, ref, semiring, f"local sort offdiag n={n}")


@pytest.mark.parametrize("semiring", ["f64", "jaccard"])
def test_local_sort_sparse_groups(dev, semiring, monkeypatch):
    # 22-bit column ids sorted by two high passes (5 + 5 bits) and the local
    # pass, with the group starts taken from the passes' histograms: the ids
    # crowd into the lowest 2^20 and the top 2^12 columns, so most groups and
    # the top digits of both passes are empty
    monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
    rng = np.random.default_rng(61)
    m, n = 20000, 1 << 22
    c = np.where(rng.random((m, 10)) < 0.9, rng.integers(0, 1 << 20, size=(m, 10)),
                 rng.integers(n - 4096, n, size=(m, 10)))
    c.sort(axis=1)
    keep = np.ones_like(c, dtype=bool)
    keep[:, 1:] = c[:, 1:] != c[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(keep.sum(axis=1))
    ci = c[keep].astype(np.int32)
    A = CSR(m, n, rp, ci, rng.random(len(ci)) + 0.5)
    run_lower(A, semiring, dev, "local sort, sparse groups")
    B = _rows_csr(rng, 3000, n, 5)
    vdt = VDT[semiring]
    O = sp.offdiag(upload(B, semiring, dev), upload(A, semiring, dev), semiring)
    ref = oracle.offdiag(B.with_values(None if vdt is None else B.values.astype(vdt)),
                         A.with_values(None if vdt is None else A.values.astype(vdt)), semiring)
    compare_full(O, ref, semiring, "local sort, sparse groups, offdiag")


@pytest.mark.parametrize("semiring", ["f64", "jaccard"])
def test_local_sort_large_groups(dev, semiring, monkeypatch):
    # groups past the first launch's LDS capacity (2048 records): 2^22
    # columns and about 6.3 M entries give 4096 groups of 1024 columns
    # (high bits max(22 - 12, bit width of 6.3 M / 2048) = 12); the entries
    # fill only the even groups, so each of those 2048 holds about 3100
    # records (more than the 1024 workgroups of the second launch, which
    # sorts them in LDS), and groups 2 and 6 take about 63000 each (sorted
    # over global memory)
    monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
    rng = np.random.default_rng(65)
    m, per, n = 630000, 10, 1 << 22
    g = 2 * rng.integers(0, 2048, size=(m, per))
    g = np.where(rng.random((m, per)) < 0.02, rng.choice([2, 6], size=(m, per)), g)
    c = np.sort(g * 1024 + rng.integers(0, 1024, size=(m, per)), axis=1)
    keep = np.ones_like(c, dtype=bool)
    keep[:, 1:] = c[:, 1:] != c[:, :-1]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(keep.sum(axis=1))
    ci = c[keep].astype(np.int32)
    A = CSR(m, n, rp, ci, rng.random(len(ci)) + 0.5)
    counts = np.bincount(ci >> 10, minlength=4096)
    assert counts[1::2].sum() == 0 and (counts[0::2] > 2048).all() and counts[2] > 4096 and counts[6] > 4096
    run_lower(A, semiring, dev, "local sort, groups past the LDS capacity")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_local_sort_group_size_limits(dev, semiring, monkeypatch):
    # 2^15 columns and under 16384 entries give 8 groups of 4096 columns
    # (high bits max(15 - 12, bit width of nnz / 2048) = 3), filled with
    # exactly 2048, 2049, 4096, 4097, 1, 0, 0 and 7 records: the limits of
    # the first launch's LDS (2048), of the second's (4096), and tiny groups;
    # off the diagonal the plus-times records carry their values
    monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
    rng = np.random.default_rng(71)
    sizes = [2048, 2049, 4096, 4097, 1, 0, 0, 7]
    cols = np.concatenate([g * 4096 + rng.integers(0, 4096, size=k) for g, k in enumerate(sizes)])
    rng.shuffle(cols)
    per = 6
    rows = [cols[i:i + per].copy() for i in range(0, len(cols), per)]
    for r in rows:  # distinct columns within a row, each redrawn inside its own group
        while len(np.unique(r)) < len(r):
            _, first = np.unique(r, return_index=True)
            dup = np.setdiff1d(np.arange(len(r)), first)
            r[dup] = (r[dup] // 4096) * 4096 + rng.integers(0, 4096, size=len(dup))
        r.sort()
    rp = np.zeros(len(rows) + 1, dtype=np.int64)
    rp[1:] = np.cumsum([len(r) for r in rows])
    ci = np.concatenate(rows).astype(np.int32)
    assert list(np.bincount(ci >> 12, minlength=8)) == sizes
    A = CSR(len(rows), 1 << 15, rp, ci, rng.random(len(ci)) + 0.5)
    run_lower(A, semiring, dev, "local sort, groups at the LDS limits")
    B = _rows_csr(rng, 500, 1 << 15, 5)
    vdt = VDT[semiring]
    O = sp.offdiag(upload(B, semiring, dev), upload(A, semiring, dev), semiring)
    compare_full(O, oracle.offdiag(B.with_values(None if vdt is None else B.values.astype(vdt)),
                                   A.with_values(None if vdt is None else A.values.astype(vdt)), semiring),
                 semiring, "local sort, groups at the LDS limits, offdiag")


@pytest.mark.parametrize("semiring", ["f64", "count"])
def test_row_longer_than_the_tile_table(dev, semiring):
    # a row of 250000 entries spans 82 tiles of 3072 entries; the
    # validation's table of tile rows (which the column sort and the row
    # products reuse) leaves the tiles deep inside it out, and those tiles
    # find their rows by search
    rng = np.random.default_rng(63)
    n = 1 << 20
    long_cols = np.sort(rng.choice(n, size=250000, replace=False)).astype(np.int32)
    B = _rows_csr(rng, 3000, n, 5)
    ci = np.concatenate([B.col_idx[: B.row_ptr[1500]], long_cols, B.col_idx[B.row_ptr[1500]:]])
    rp = np.concatenate([B.row_ptr[:1501], B.row_ptr[1500:] + 250000]).astype(np.int64)
    A = CSR(3001, n, rp, ci, rng.random(len(ci)) + 0.5)
    run_lower(A, semiring, dev, "a row longer than 64 tiles")


WORKLOADS = [("tiny_uniform_f64", 0), ("kmer_i32", 5), ("rmat20_f32", 7), ("jaccard_large", 7),
             ("offdiag_f64", 5)]


@pytest.mark.parametrize("name,shift", WORKLOADS)
def test_workloads_reduced(dev, name, shift):
    w = W.make(name, 1, shift)
    A = w["A"]
    sr = w["semiring"]
    C = run_lower(A, sr, dev, f"{name}>>{shift}")
    if "mirror" in w["ops"]:
        # the device's C_L mirrored, against the oracle's own C_L mirrored (the
        # workloads' values are positive: the entries' bar is relative)
        M = sp.mirror(C, sr)
        L = oracle.lower(A.with_values(A.values.astype(VDT[sr]) if VDT[sr] else None), sr)
        ref = oracle.mirror(A.nrows, L.row_ptr, L.col_idx, L.values)
        compare_full(M, ref, "count" if sr == "count" else sr, f"{name} mirror")
    if "offdiag" in w["ops"]:
        Ai, Aj = w["A"], w["B"]
        O = sp.offdiag(upload(Ai, sr, dev), upload(Aj, sr, dev), sr)
        compare_full(O, oracle.offdiag(Ai, Aj, sr), sr, f"{name} offdiag")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_offdiag_random(dev, semiring):
    rng = np.random.default_rng(31)
    for t in range(6):
        mi, mj, n = int(rng.integers(1, 200)), int(rng.integers(1, 200)), int(rng.integers(1, 300))
        Ai = random_csr(rng, mi, n, 0.04, signed=True)
        Aj = random_csr(rng, mj, n, 0.04, signed=True)
        if VDT[semiring] is not None:
            Ai = Ai.with_values(Ai.values.astype(VDT[semiring]))
            Aj = Aj.with_values(Aj.values.astype(VDT[semiring]))
        O = sp.offdiag(upload(Ai, semiring, dev), upload(Aj, semiring, dev), semiring)
        compare_full(O, oracle.offdiag(Ai if VDT[semiring] else Ai.with_values(None),
                                       Aj if VDT[semiring] else Aj.with_values(None), semiring),
                     semiring, f"offdiag case {t}")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_offdiag_half(dev, semiring):
    # Algorithm 3's half blocks: odd and even row counts, a single row (empty
    # top half), an empty operand, and enough rows for several tiles
    rng = np.random.default_rng(43)
    vdt = VDT[semiring]
    for t, (mi, mj, n) in enumerate([(37, 23, 60), (1, 5, 10), (2, 1, 10), (0, 4, 7), (3001, 2999, 4000)]):
        Ai = random_csr(rng, mi, n, 0.01 if mi > 100 else 0.1, signed=True)
        Aj = random_csr(rng, mj, n, 0.01 if mj > 100 else 0.1, signed=True)
        if vdt is not None:
            Ai, Aj = Ai.with_values(Ai.values.astype(vdt)), Aj.with_values(Aj.values.astype(vdt))
        else:
            Ai, Aj = Ai.with_values(None), Aj.with_values(None)
        for half in ("top", "right"):
            print(f"[offdiag_half {semiring}] case {t} {half} mi={mi} mj={mj}", flush=True)
            O = sp.offdiag_half(upload(Ai, semiring, dev), upload(Aj, semiring, dev), half, semiring)
            assert (O.nrows, O.ncols) == ((mi // 2 if half == "top" else mi), mj)
            compare_full(O, oracle.offdiag_half(Ai, Aj, half, semiring), semiring, f"half {half} case {t}")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_offdiag_self_product(dev, semiring):
    # offdiag(A, A): every row meets itself in each of its columns, so the
    # diagonal entry merges as many terms as the row has entries (buckets of
    # 1 to 90 products: the small, one-per-lane and whole-bucket merges)
    rng = np.random.default_rng(45)
    vdt = VDT[semiring]
    m, n = 600, 20000  # (few entries per column: the rows stay light)
    lens = rng.integers(0, 91, size=m)
    rows = [np.sort(rng.choice(n, size=int(k), replace=False)) for k in lens]
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum(lens)
    ci = np.concatenate(rows).astype(np.int32)
    A = CSR(m, n, rp, ci, rng.standard_normal(len(ci)))
    Ah = A.with_values(A.values.astype(vdt) if vdt is not None else None)
    print(f"[offdiag self {semiring}] m={m} nnz={A.nnz}", flush=True)
    O = sp.offdiag(upload(A, semiring, dev), upload(A, semiring, dev), semiring)
    compare_full(O, oracle.offdiag(Ah, Ah, semiring), semiring, "offdiag(A, A)")


def test_offdiag_halves_cover_on_device(dev, monkeypatch):
    # the top half of C_ij and the transposed right half of C_ji rebuild the
    # device's own full block bit for bit; the second case takes the column
    # sort's local path (2^20 columns), where the right operand's arrays start
    # at an entry offset
    import torch
    import scipy.sparse as ssp
    rng = np.random.default_rng(44)
    for case, (mi, mj, n, local) in enumerate([(301, 199, 500, False), (3001, 2001, 1 << 20, True)]):
        if local:
            monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
        if local:
            Ai, Aj = _rows_csr(rng, mi, n, 5), _rows_csr(rng, mj, n, 5)
        else:
            Ai, Aj = random_csr(rng, mi, n, 0.02), random_csr(rng, mj, n, 0.02)
        full = sp.offdiag(upload(Ai, "f64", dev), upload(Aj, "f64", dev), "f64")
        top = sp.offdiag_half(upload(Ai, "f64", dev), upload(Aj, "f64", dev), "top", "f64")
        right = sp.offdiag_half(upload(Aj, "f64", dev), upload(Ai, "f64", dev), "right", "f64")
        frp, fci, fv = full.to_host()
        trp, tci, tv = top.to_host()
        rrp, rci, rv = right.to_host()
        cut = frp[mi // 2]
        np.testing.assert_array_equal(trp, frp[:mi // 2 + 1])
        np.testing.assert_array_equal(tci, fci[:cut])
        np.testing.assert_array_equal(tv.view(np.uint64), fv[:cut].view(np.uint64))
        R = ssp.csr_matrix((rv, rci, rrp), shape=(mj, mi)).T.tocsr()
        R.sort_indices()
        assert R.indptr[mi // 2] == 0
        np.testing.assert_array_equal(R.indptr[mi // 2:], frp[mi // 2:] - cut)
        np.testing.assert_array_equal(R.indices, fci[cut:])
        # (the same products, summed over k in the same order on both sides)
        np.testing.assert_allclose(R.data, fv[cut:], rtol=1e-12, atol=0)


SYMM_TOL = {"f64": 1e-12, "count": 1e-12, "jaccard": 2.0 ** -24, "f32": 1e-5 + 2.0 ** -24}


def _symm_ref(L, X):
    """The oracle's Y and its tolerance scale: sum over the terms of
    |C_L entry scale| |x|, where an entry's scale is the sum of |products|
    behind it (C_L on the device agrees with the oracle's to the lower
    product's bar: bit for bit for counts and Jaccard, 1e-12 / 1e-5 of that
    sum for f64 / f32), and Y is rounded once from double."""
    m = L.nrows
    ref, _ = oracle.symm(m, L.row_ptr, L.col_idx, L.values, X)
    ent = L.sum_abs if L.sum_abs is not None else np.abs(L.values.astype(np.float64))
    scale, _ = oracle.symm(m, L.row_ptr, L.col_idx, ent, np.abs(X))
    return ref, np.maximum(scale, np.abs(ref))


def _hcat(A1, A2):
    D1 = np.zeros((A1.nrows, A1.ncols)); P1 = np.zeros_like(D1, dtype=bool)
    D2 = np.zeros((A2.nrows, A2.ncols)); P2 = np.zeros_like(D2, dtype=bool)
    for A, D, P in ((A1, D1, P1), (A2, D2, P2)):
        r = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
        D[r, A.col_idx] = A.values
        P[r, A.col_idx] = True
    return csr_from_dense(np.hstack([D1, D2]), pattern=np.hstack([P1, P2]))


@pytest.mark.parametrize("semiring", ["f64", "f32", "count"])
def test_lower_accumulate(dev, semiring):
    # stage accumulation against the oracle, starting from an empty sum and
    # from a previous stage; rows of several wavefront lengths
    rng = np.random.default_rng(47)
    vdt = VDT[semiring]
    m = 500
    A1 = random_csr(rng, m, 300, 0.03, signed=True)
    A2 = random_csr(rng, m, 200, 0.05, signed=True)
    cast = (lambda A: A.with_values(A.values.astype(vdt))) if vdt is not None else (lambda A: A.with_values(None))
    empty = sp.DeviceCSR.from_host(CSR(m, m, np.zeros(m + 1, np.int64), np.zeros(0, np.int32),
                                       np.zeros(0, dtype={"f64": np.float64, "f32": np.float32,
                                                          "count": np.int32}[semiring])), dev)
    print(f"[accumulate {semiring}] m={m}", flush=True)
    C1 = sp.lower_accumulate(empty, upload(A1, semiring, dev), semiring)
    R1 = oracle.lower(cast(A1), semiring)
    compare_full(C1, R1, semiring, "first stage")
    C2 = sp.lower_accumulate(C1, upload(A2, semiring, dev), semiring)
    R2 = oracle.lower_accumulate(R1, cast(A2), semiring)
    compare_full(C2, R2, semiring, "second stage")
    # the same as the lower part of the concatenated stages (structure exactly)
    L = sp.lower(upload(_hcat(A1, A2), semiring, dev), semiring)
    rp2, ci2, _ = C2.to_host()
    rpl, cil, _ = L.to_host()
    np.testing.assert_array_equal(rp2, rpl)
    np.testing.assert_array_equal(ci2, cil)


def _chunk_case(rng, m, n, hub_rows):
    # sparse rows, a hub column shared by hub_rows rows (their lower rows grow
    # past what a chunk of the merge holds), 2600 consecutive empty rows (more
    # than a chunk's row limit) and a few more empty rows
    D = rng.random((m, n)) < 0.002
    D[2000:4600] = False
    D[rng.choice(m, size=hub_rows, replace=False), 0] = True
    D[rng.choice(m, size=40, replace=False), :] = False
    return csr_from_dense(np.where(D, rng.standard_normal((m, n)), 0.0), pattern=D)


@pytest.mark.parametrize("semiring", ["f64", "f32", "count"])
def test_lower_accumulate_chunks(dev, semiring):
    # the merge's chunks of rows: long rows alone in a chunk (up to 3000
    # entries of the two parts), chunks cut by the row limit, empty rows
    rng = np.random.default_rng(49)
    vdt = VDT[semiring]
    cast = (lambda A: A.with_values(A.values.astype(vdt))) if vdt is not None else (lambda A: A.with_values(None))
    A1, A2 = _chunk_case(rng, 6000, 300, 1500), _chunk_case(rng, 6000, 300, 1500)
    print(f"[accumulate chunks {semiring}] m=6000", flush=True)
    R1 = oracle.lower(cast(A1), semiring)
    C1 = sp.lower(upload(A1, semiring, dev), semiring)
    C2 = sp.lower_accumulate(C1, upload(A2, semiring, dev), semiring)
    compare_full(C2, oracle.lower_accumulate(R1, cast(A2), semiring), semiring, "chunks")


def _with_long_rows(rng, m, n):
    # short random rows plus a few long ones (heavy rows: many products)
    A = _rows_csr(rng, m, n, 6)
    D = np.zeros((m, n), dtype=bool)
    r = np.repeat(np.arange(m), np.diff(A.row_ptr))
    D[r, A.col_idx] = True
    for i in rng.choice(m, size=6, replace=False):
        D[i, rng.choice(n, size=min(n, 400), replace=False)] = True
    return csr_from_dense(np.where(D, rng.random((m, n)) + 0.5, 0.0), pattern=D)


@pytest.mark.parametrize("semiring", SEMIRINGS)
@pytest.mark.parametrize("local", [False, True])
def test_plan_execute(dev, semiring, local, monkeypatch):
    # the two-phase use: a plan from one set of values, executions with new
    # values of the same pattern; each equals the one-shot product of those
    # values (bit for bit for counts and Jaccard) and the oracle to the usual
    # bar.  local: the column
    # sort's local path (the entry behind each index position comes from it)
    import torch
    if local:
        monkeypatch.setenv("SPSYRK_LOCAL_SORT", "1")
    rng = np.random.default_rng(49)
    vdt = VDT[semiring]
    A = _with_long_rows(rng, 900, 1200)
    print(f"[plan {semiring} local={local}] m={A.nrows} nnz={A.nnz}", flush=True)
    plan, C0 = sp.lower_plan(upload(A, semiring, dev), semiring)
    compare_full(C0, oracle.lower(A.with_values(A.values.astype(vdt) if vdt else None), semiring), semiring, "plan")
    assert sp.stats()["heavy_rows"] > 0
    for t in range(2):
        B = A.with_values(rng.standard_normal(A.nnz))
        Bd = upload(B, semiring, dev)
        E = plan.execute(Bd.values)
        L = sp.lower(Bd, semiring)
        assert E.nnz == L.nnz
        assert torch.equal(E.row_ptr, L.row_ptr)
        assert torch.equal(E.col_idx[: E.nnz], L.col_idx[: L.nnz])
        if vdt is None:  # (plus-times sums of heavy rows may end in other bits from run to run)
            assert torch.equal(E.values[: E.nnz].view(torch.uint8), L.values[: L.nnz].view(torch.uint8))
        compare_full(E, oracle.lower(B.with_values(B.values.astype(vdt) if vdt else None), semiring), semiring,
                     f"execute {t}")
    plan.close()


@pytest.mark.parametrize("semiring", SEMIRINGS)
@pytest.mark.parametrize("radix", ["3", "9", "1"])
def test_packed_run_lengths(dev, semiring, radix, monkeypatch):
    # partner runs packed with radix 3 or 9 (runs of 2 or 8 partners and
    # longer escape to the full table) or all in the full table (1): lower on
    # both column-sort paths with heavy rows, off-diagonal, and a plan's
    # executions all match the oracle
    monkeypatch.setenv("SPSYRK_RUN_RADIX", radix)
    rng = np.random.default_rng(53)
    vdt = VDT[semiring]
    A = _with_long_rows(rng, 700, 900)
    for local in ("0", "1"):
        monkeypatch.setenv("SPSYRK_LOCAL_SORT", local)
        print(f"[packed runs {semiring} radix={radix} local={local}] m={A.nrows} nnz={A.nnz}", flush=True)
        run_lower(A, semiring, dev, f"packed runs radix={radix} local={local}")
        assert sp.stats()["heavy_rows"] > 0
        B = _rows_csr(rng, 300, 900, 6)
        B = B.with_values(B.values.astype(vdt) if vdt else None)
        Av = A.with_values(A.values.astype(vdt) if vdt else None)
        O = sp.offdiag(upload(A, semiring, dev), upload(B, semiring, dev), semiring)
        compare_full(O, oracle.offdiag(Av, B, semiring), semiring, f"packed runs offdiag radix={radix}")
    plan, C0 = sp.lower_plan(upload(A, semiring, dev), semiring)
    E = plan.execute(upload(A, semiring, dev).values)
    compare_full(E, oracle.lower(A.with_values(A.values.astype(vdt) if vdt else None), semiring), semiring,
                 f"packed runs plan radix={radix}")
    plan.close()


@pytest.mark.parametrize("semiring", ["count", "jaccard"])
@pytest.mark.parametrize("pack", ["1", "0"])
def test_packed_staging(dev, semiring, pack, monkeypatch):
    # counts and Jaccard values of the light rows staged as one packed word
    # (on where it fits) or as column and value (off); a matrix with a
    # 300-entry row over 100000 rows is too wide for the words and takes the
    # plain staging either way
    monkeypatch.setenv("SPSYRK_PACK_STAGING", pack)
    rng = np.random.default_rng(59)
    for m, n, per in ((3000, 400, 6), (20000, 1 << 20, 12)):
        A = _rows_csr(rng, m, n, per)
        run_lower(A, semiring, dev, f"packed staging {pack} m={m}")
    # row 0 replaced by 300 columns
    A = _rows_csr(rng, 100000, 1 << 16, 3)
    long_cols = np.sort(rng.choice(1 << 16, size=300, replace=False)).astype(np.int32)
    ci = np.concatenate([long_cols, A.col_idx[A.row_ptr[1]:]])
    rp = np.concatenate([[0], A.row_ptr[1:] - A.row_ptr[1] + 300]).astype(np.int64)
    W = CSR(A.nrows, A.ncols, rp, ci, np.ones(len(ci)))
    run_lower(W, semiring, dev, f"packed staging {pack} with a 300-entry row")


@pytest.mark.parametrize("semiring", ["f64", "jaccard"])
@pytest.mark.parametrize("rows", ["32", "8", "1"])
def test_rows_per_chunk(dev, semiring, rows, monkeypatch):
    # the light kernel's chunks of 32 rows (large matrices), 8 (small ones)
    # and 1, forced on a matrix with heavy rows: lower and off-diagonal
    # products match the oracle
    monkeypatch.setenv("SPSYRK_ROWS_PER_CHUNK", rows)
    rng = np.random.default_rng(67)
    vdt = VDT[semiring]
    A = _with_long_rows(rng, 1500, 1200)
    run_lower(A, semiring, dev, f"{rows} rows per chunk")
    assert sp.stats()["heavy_rows"] > 0
    B = _rows_csr(rng, 700, 1200, 5)
    O = sp.offdiag(upload(A, semiring, dev), upload(B, semiring, dev), semiring)
    compare_full(O, oracle.offdiag(A.with_values(A.values.astype(vdt) if vdt else None),
                                   B.with_values(B.values.astype(vdt) if vdt else None), semiring), semiring,
                 f"{rows} rows per chunk offdiag")


def test_plan_of_empty_matrix(dev):
    A = CSR(5, 7, np.zeros(6, np.int64), np.zeros(0, np.int32), np.zeros(0))
    plan, C = sp.lower_plan(upload(A, "f64", dev), "f64")
    E = plan.execute(upload(A, "f64", dev).values)
    assert C.nnz == 0 and E.nnz == 0 and E.nrows == 5
    plan.close()


def test_lower_accumulate_rejects_jaccard(dev):
    A = random_csr(np.random.default_rng(48), 10, 10, 0.3)
    C = sp.lower(upload(A, "jaccard", dev), "jaccard")
    with pytest.raises(sp.SpsyrkError):
        sp.lower_accumulate(C, upload(A, "jaccard", dev), "jaccard")


def _check_symm(Y, ref, scale, semiring, what):
    err = np.abs(Y.astype(np.float64) - ref)
    bad = err > SYMM_TOL[semiring] * scale + 1e-300
    assert not bad.any(), f"{what}: {int(bad.sum())} elements out of tolerance, max err {float(err.max())!r}"


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_symm_matches_oracle(dev, semiring):
    # Y = C X from C_L only (Eq. (spmv), (spgemm)): 1, 3, 8 and 11 columns (the
    # column blocks of 8, 2 and 1), a padded leading dimension, empty rows
    import torch
    rng = np.random.default_rng(46)
    vdt = VDT[semiring]
    xdt = np.float64 if semiring in ("f64", "count") else np.float32
    A = random_csr(rng, 700, 900, 0.01, signed=True)
    Ah = A.with_values(A.values.astype(vdt) if vdt is not None else None)
    C = sp.lower(upload(A, semiring, dev), semiring)
    L = oracle.lower(Ah, semiring)
    for k in (1, 3, 8, 11):
        print(f"[symm {semiring}] k={k}", flush=True)
        X = rng.standard_normal((A.nrows, k + 2)).astype(xdt)
        Xd = torch.from_numpy(X).to(dev)[:, :k]  # row stride k + 2
        Y = sp.symm(C, Xd, semiring).cpu().numpy()
        ref, scale = _symm_ref(L, X[:, :k].astype(np.float64))
        _check_symm(Y, ref, scale, semiring, f"symm k={k}")
    # a vector
    x = rng.standard_normal(A.nrows).astype(xdt)
    y = sp.symm(C, torch.from_numpy(x).to(dev), semiring).cpu().numpy()
    ref, scale = _symm_ref(L, x.astype(np.float64)[:, None])
    _check_symm(y[:, None], ref, scale, semiring, "symm vector")


@pytest.mark.parametrize("semiring,bits", [("f64", "12"), ("f32", "13"), ("count", "14"), ("jaccard", "12"),
                                           ("f64", "0")])
def test_symm_vector_buckets(dev, semiring, bits, monkeypatch):
    # the product with one column with its transposed term bucketed (forced at
    # this size; buckets of 2^12 to 2^14 rows, so 3 to 1 of them), several
    # counting workgroups and summing parts, empty rows; and with buckets off
    import torch
    monkeypatch.setenv("SPSYRK_SYMM_BUCKETS", bits)
    rng = np.random.default_rng(50)
    vdt = VDT[semiring]
    xdt = np.float64 if semiring in ("f64", "count") else np.float32
    A = _rows_csr(rng, 12000, 4000, 5)
    A = A.with_values(rng.standard_normal(A.nnz))
    keep = np.ones(A.nrows, dtype=bool)
    keep[rng.choice(A.nrows, size=300, replace=False)] = False
    D = np.zeros(A.nrows + 1, dtype=np.int64)
    lens = np.diff(A.row_ptr) * keep
    np.cumsum(lens, out=D[1:])
    sel = np.repeat(keep, np.diff(A.row_ptr))
    A = CSR(A.nrows, A.ncols, D, A.col_idx[sel], A.values[sel])
    Ah = A.with_values(A.values.astype(vdt) if vdt is not None else None)
    C = sp.lower(upload(A, semiring, dev), semiring)
    L = oracle.lower(Ah, semiring)
    print(f"[symm buckets {semiring} {bits}] m={A.nrows} nnz_L={L.nnz}", flush=True)
    assert L.nnz > 3 * 65536
    x = rng.standard_normal(A.nrows).astype(xdt)
    y = sp.symm(C, torch.from_numpy(x).to(dev), semiring).cpu().numpy()
    ref, scale = _symm_ref(L, x.astype(np.float64)[:, None])
    _check_symm(y[:, None], ref, scale, semiring, "symm buckets")


@pytest.mark.parametrize("semiring,bits", [("f64", "10"), ("f32", "11"), ("count", "10"), ("jaccard", "12"),
                                           ("f64", "0")])
def test_symm_vector_split(dev, semiring, bits, monkeypatch):
    # the product with one column with its transposed term written as records
    # grouped by row ranges and added range by range (forced at this size:
    # ranges of 2^10 to 2^12 rows, so 12 to 3 of them and, at 2^10, two launches
    # of eight ranges; "0": one range of 2^18 rows), empty rows
    import torch
    monkeypatch.setenv("SPSYRK_SYMM_SPLIT", "1")
    monkeypatch.setenv("SPSYRK_SYMM_BUCKETS", "0")
    monkeypatch.setenv("SPSYRK_SYMM_SPLIT_BITS", bits)
    rng = np.random.default_rng(51)
    vdt = VDT[semiring]
    xdt = np.float64 if semiring in ("f64", "count") else np.float32
    A = _rows_csr(rng, 12000, 4000, 5)
    A = A.with_values(rng.standard_normal(A.nnz))
    keep = np.ones(A.nrows, dtype=bool)
    keep[rng.choice(A.nrows, size=300, replace=False)] = False
    D = np.zeros(A.nrows + 1, dtype=np.int64)
    np.cumsum(np.diff(A.row_ptr) * keep, out=D[1:])
    sel = np.repeat(keep, np.diff(A.row_ptr))
    A = CSR(A.nrows, A.ncols, D, A.col_idx[sel], A.values[sel])
    Ah = A.with_values(A.values.astype(vdt) if vdt is not None else None)
    C = sp.lower(upload(A, semiring, dev), semiring)
    L = oracle.lower(Ah, semiring)
    print(f"[symm split {semiring} {bits}] m={A.nrows} nnz_L={L.nnz}", flush=True)
    x = rng.standard_normal(A.nrows).astype(xdt)
    y = sp.symm(C, torch.from_numpy(x).to(dev), semiring).cpu().numpy()
    ref, scale = _symm_ref(L, x.astype(np.float64)[:, None])
    _check_symm(y[:, None], ref, scale, semiring, "symm split")


def test_symm_rejects_upper_entries(dev):
    import torch
    P = csr_from_dense(np.array([[1.0, 2.0], [0.0, 3.0]]))
    with pytest.raises(sp.SpsyrkError):
        sp.symm(sp.DeviceCSR.from_host(P, dev), torch.ones(2, dtype=torch.float64, device=dev), "f64")


@pytest.mark.parametrize("semiring", SEMIRINGS)
def test_mirror_matches_oracle(dev, semiring):
    rng = np.random.default_rng(77)
    A = random_csr(rng, 400, 600, 0.02, signed=False)
    C = sp.lower(upload(A, semiring, dev), semiring)
    M = sp.mirror(C, semiring)
    vdt = VDT[semiring]
    L = oracle.lower(A.with_values(A.values.astype(vdt) if vdt is not None else None), semiring)
    ref = oracle.mirror(A.nrows, L.row_ptr, L.col_idx, L.values)
    compare_full(M, ref, "count" if semiring == "count" else semiring, "mirror")
    # offdiag(A, A) is the full product: same structure as the mirror
    O = sp.offdiag(upload(A, semiring, dev), upload(A, semiring, dev), semiring)
    np.testing.assert_array_equal(O.to_host()[0], M.to_host()[0])
    np.testing.assert_array_equal(O.to_host()[1], M.to_host()[1])


def _random_lower(rng, m, per_row, hub):
    # lower-triangular CSR: about per_row random columns below the diagonal,
    # the hub column in every row past it, the diagonal in every other row
    rows_c = []
    for i in range(m):
        c = set(rng.integers(0, i, size=min(per_row, i)).tolist()) if i > 0 else set()
        if i > hub:
            c.add(hub)
        if i % 2 == 0:
            c.add(i)
        rows_c.append(sorted(c))
    rp = np.zeros(m + 1, dtype=np.int64)
    rp[1:] = np.cumsum([len(c) for c in rows_c])
    ci = np.array([x for c in rows_c for x in c], dtype=np.int32)
    return rp, ci, rng.standard_normal(len(ci))


@pytest.mark.parametrize("cap", [1, 700, 5000])
def test_mirror_column_slabs(dev, cap, monkeypatch):
    # the transpose in many column slabs (slab size lowered from 2^31 records),
    # a hub column holding more records than a slab, and histogram buckets
    # over the slab size split by finer histograms of their columns
    monkeypatch.setenv("SPSYRK_MIRROR_SLAB", str(cap))
    rng = np.random.default_rng(cap)
    m = 300 if cap == 1 else 9000
    rp, ci, v = _random_lower(rng, m, 12, 5)
    print(f"[mirror slabs] cap={cap} m={m} nnz={len(ci)}", flush=True)
    ref = oracle.mirror(m, rp, ci, v)
    M = sp.mirror(_raw(dev, rp, ci, m, v), "f64")
    compare_full(M, ref, "f64", f"mirror slabs {cap}")
    M = sp.mirror(_raw(dev, rp, ci, m, None), "count")
    np.testing.assert_array_equal(M.to_host()[0], ref.row_ptr)
    np.testing.assert_array_equal(M.to_host()[1], ref.col_idx)


@pytest.mark.parametrize("bits,cap,m", [(4, 1 << 31, 5000), (8, 1 << 31, 5000), (10, 3000, 5000),
                                        (0, 1 << 31, 70000)])
@pytest.mark.parametrize("direct", ["0", "1"])
def test_mirror_narrow_slabs(dev, bits, cap, m, direct, monkeypatch):
    # slabs of at most 2^bits columns (keys of at most 16 bits: one or two
    # sort passes, the first over extracted records or reading C_L through
    # the slab's rows (direct), the last placing into the full rows), with
    # and without the record cap; the slab plan's histogram counts every
    # entry by column and takes the diagonal off again.  bits 0: one slab of
    # 70000 columns, 17-bit keys, sorted over extracted records and placed
    # by a pass of its own
    monkeypatch.setenv("SPSYRK_MIRROR_NARROW", str(bits))
    monkeypatch.setenv("SPSYRK_MIRROR_SLAB", str(cap))
    monkeypatch.setenv("SPSYRK_SLAB_DIRECT", direct)
    rng = np.random.default_rng(bits)
    rp, ci, v = _random_lower(rng, m, 20 if m < 10000 else 4, 7)
    print(f"[mirror narrow] bits={bits} cap={cap} m={m} nnz={len(ci)}", flush=True)
    ref = oracle.mirror(m, rp, ci, v)
    M = sp.mirror(_raw(dev, rp, ci, m, v), "f64")
    compare_full(M, ref, "f64", f"mirror narrow {bits}")
    M = sp.mirror(_raw(dev, rp, ci, m, v.astype(np.float32)), "f32")
    np.testing.assert_array_equal(M.to_host()[0], ref.row_ptr)
    np.testing.assert_array_equal(M.to_host()[1], ref.col_idx)


def test_mirror_structure_only(dev):
    import torch
    rng = np.random.default_rng(5)
    A = random_csr(rng, 100, 80, 0.05)
    C = sp.lower(upload(A, "count", dev), "count")
    C_nov = sp.DeviceCSR(C.nrows, C.ncols, C.row_ptr, C.col_idx, None, C.nnz)
    M = sp.mirror(C_nov, "count")
    assert M.values is None
    L = oracle.lower(A.with_values(None), "count")
    ref = oracle.mirror(A.nrows, L.row_ptr, L.col_idx, L.values)
    np.testing.assert_array_equal(M.to_host()[0], ref.row_ptr)
    np.testing.assert_array_equal(M.to_host()[1], ref.col_idx)
    del torch


def test_phase_timing(dev):
    # every phase timed, then only the light numeric phase: the selection
    # records that phase alone, once per call, and the product is unchanged
    A = W.make("kmer_i32", 1, 6)["A"]
    Ad = upload(A, "count", dev)
    sp.timing_begin()
    X = sp.lower(Ad, "count").to_host()
    ph = sp.timing_end()
    assert {"validate", "colindex", "runs", "light_numeric", "compact"} <= set(ph)
    sp.timing_begin(["light_numeric"])
    Y = sp.lower(Ad, "count").to_host()
    Y2 = sp.lower(Ad, "count").to_host()
    ph = sp.timing_end()
    assert set(ph) == {"light_numeric"} and ph["light_numeric"][1] == 2 and ph["light_numeric"][0] > 0
    sp.timing_begin([])
    sp.lower(Ad, "count")
    assert sp.timing_end() == {}
    for a, b, c in zip(X, Y, Y2):
        np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(a, c)


def test_deterministic(dev):
    A = W.make("kmer_i32", 1, 6)["A"]
    X = sp.lower(upload(A, "count", dev), "count").to_host()
    Y = sp.lower(upload(A, "count", dev), "count").to_host()
    for a, b in zip(X, Y):
        np.testing.assert_array_equal(a, b)


def _raw(dev, rp, ci, n, vals=None):
    import torch
    return sp.DeviceCSR(len(rp) - 1, n, torch.tensor(rp, dtype=torch.int64, device=dev),
                        torch.tensor(ci, dtype=torch.int32, device=dev),
                        None if vals is None else torch.tensor(vals, device=dev), rp[-1])


def test_rejects_non_canonical_on_device(dev):
    bad = [
        ([0, 2, 3], [1, 0, 2], 4),   # unsorted row
        ([0, 2, 3], [1, 1, 2], 4),   # duplicate column
        ([0, 2, 3], [1, 7, 2], 4),   # column out of range
        ([0, 3, 2], [1, 2, 3], 4),   # row_ptr decreasing
    ]
    for rp, ci, n in bad:
        with pytest.raises(sp.SpsyrkError) as ei:
            sp.lower(_raw(dev, rp, ci, n, np.ones(len(ci))), "f64")
        assert ei.value.status == 2
    with pytest.raises(sp.SpsyrkError) as ei:   # entry above the diagonal
        sp.mirror(_raw(dev, [0, 2, 3], [0, 1, 0], 2, np.ones(3)), "f64")
    assert ei.value.status == 2
    # off the diagonal both operands' flags are read at once; the message
    # names the operand that failed (the left one first)
    good = _raw(dev, [0, 2, 3], [1, 2, 3], 4, np.ones(3))
    for rp, ci, n in bad:
        for left in (True, False):
            B = _raw(dev, rp, ci, n, np.ones(len(ci)))
            with pytest.raises(sp.SpsyrkError) as ei:
                sp.offdiag(B, good, "f64") if left else sp.offdiag(good, B, "f64")
            assert ei.value.status == 2 and ("Ai" if left else "Aj") in ei.value.detail
    with pytest.raises(sp.SpsyrkError) as ei:
        sp.offdiag(_raw(dev, [0, 2, 3], [1, 0, 2], 4, np.ones(3)), _raw(dev, [0, 2, 3], [1, 7, 2], 4, np.ones(3)),
                   "f64")
    assert ei.value.status == 2 and "Ai" in ei.value.detail
    np.testing.assert_array_equal(sp.offdiag(good, good, "f64").to_host()[0], [0, 1, 2])
