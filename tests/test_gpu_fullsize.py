"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times.  The k-mer, Jaccard and off-diagonal workloads are compared
with the oracle row for row over every row (the oracle's rows computed in
blocks on all host threads); R-MAT's much larger result is compared on sampled
rows.  Whole-result properties that hold at any size are checked on the device
output too (exact count sums, diagonal, entry counts, symmetry of sampled
mirrored rows)."""
import functools

import numpy as np
import pytest

import oracle
import paper_2608_09713_amd as sp
from paper_2608_09713_amd import workloads as W
from tests.parity import compare_full, compare_rows, device_rows

pytestmark = pytest.mark.gpu

VDT = {"f64": np.float64, "f32": np.float32, "count": None, "jaccard": None}


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available()
    sp.library()
    return "cuda:0"


@functools.lru_cache(maxsize=8)
def make(name):
    """A full-size workload, generated once per test session."""
    return W.make(name, 1, 0)


def upload(A, sr, dev):
    vdt = VDT[sr]
    return sp.DeviceCSR.from_host(A.with_values(A.values.astype(vdt) if vdt else None), dev)


def sample_rows(A, k, seed, extra=()):
    rng = np.random.default_rng(seed)
    rows = set(int(r) for r in rng.choice(A.nrows, size=min(k, A.nrows), replace=False))
    rows.update(int(r) for r in extra)
    rows.update([0, A.nrows - 1])
    return np.array(sorted(rows), dtype=np.int64)


def col_counts(A):
    return np.bincount(A.col_idx, minlength=A.ncols).astype(np.int64)


def check_lower(A, sr, dev, rows, what):
    """C_L on the device against the oracle: every row (rows is None) or the
    listed rows."""
    print(f"[full {what}] m={A.nrows} n={A.ncols} nnz={A.nnz}", flush=True)
    C = sp.lower(upload(A, sr, dev), sr)
    st = sp.stats()
    Ain = A.with_values(A.values.astype(VDT[sr]) if VDT[sr] else None)
    if rows is None:
        ref = oracle.lower(Ain, sr, threads=oracle.host_threads())
        print(f"[full {what}] oracle done: nnz={ref.nnz}; comparing every row", flush=True)
        compare_full(C, ref, sr, what)
        del ref
    else:
        ref = oracle.lower(Ain, sr, rows=rows)
        compare_rows(C, ref, rows, sr, what)
    # entry count of every row is at least 1 for non-empty rows, the diagonal is last
    rp = C.row_ptr.cpu().numpy()
    lens = np.diff(A.row_ptr)
    ne = np.flatnonzero(lens > 0)
    assert np.all(np.diff(rp)[lens == 0] == 0)
    import torch
    last = torch.from_numpy(rp[ne + 1] - 1).to(C.col_idx.device)
    assert torch.equal(C.col_idx[last].cpu(), torch.from_numpy(ne.astype(np.int32)))
    return C, st, ne, last


@pytest.mark.parametrize("name", ["kmer_i32", "jaccard_large"])
def test_kmer_shapes_full(dev, name):
    import torch
    w = make(name)
    A, sr = w["A"], w["semiring"]
    C, st, ne, last = check_lower(A, sr, dev, None, name)
    c = col_counts(A)
    F_L = int((c * (c + 1) // 2).sum())
    assert st["products"] + A.nnz == F_L  # half-work identity: formed products = F_L exactly
    if sr == "count":
        assert int(C.values[: C.nnz].to(torch.int64).sum().item()) == F_L
        assert torch.equal(C.values[last].cpu(), torch.from_numpy(np.diff(A.row_ptr)[ne].astype(np.int32)))
    else:
        v = C.values[: C.nnz]
        assert bool(((v > 0) & (v <= 1)).all().item())
        assert bool((C.values[last] == 1.0).all().item())
        # count semiring on the same input: the Jaccard structure is the count structure
        K = sp.lower(upload(A, "count", dev), "count")
        assert K.nnz == C.nnz and torch.equal(K.row_ptr, C.row_ptr)
        assert torch.equal(K.col_idx[: K.nnz], C.col_idx[: C.nnz])
        assert int(K.values[: K.nnz].to(torch.int64).sum().item()) == F_L


def test_rmat_full_lower_and_mirror(dev):
    import torch
    w = make("rmat20_f32")
    A, sr = w["A"], w["semiring"]
    lens = np.diff(A.row_ptr)
    heavy = np.argsort(lens)[-3:]  # hub rows: the longest rows
    rows = sample_rows(A, 60, 12, extra=heavy)
    C, st, ne, last = check_lower(A, sr, dev, rows, "rmat20")
    assert st["heavy_rows"] > 0
    # diagonal = squared row norm (float64 on the host, float32 on the device)
    sq = np.add.reduceat(A.values.astype(np.float64) ** 2, A.row_ptr[ne])
    d = C.values[last].cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(d, sq, rtol=1e-6)
    nnz_L = C.nnz
    M = sp.mirror(C, sr)
    del C
    torch.cuda.empty_cache()
    assert M.nnz == 2 * nnz_L - len(ne)
    # sampled full rows: the same structure as A A^T computed directly by the oracle,
    # values within the fp32 bound; C(i, j) and C(j, i) bitwise equal
    ref = oracle.offdiag(A, A, "f32", rows=rows)
    compare_rows(M, ref, rows, "f32", "rmat20 mirror rows")
    mrp, mci, mv = device_rows(M, rows)
    rp_full = M.row_ptr.cpu().numpy()
    for q, i in enumerate(rows[:20]):
        cols = mci[mrp[q]:mrp[q + 1]]
        vals = mv[mrp[q]:mrp[q + 1]]
        js = cols[:8]
        jr, jc, jv = device_rows(M, js)
        for t, j in enumerate(js):
            seg_c = jc[jr[t]:jr[t + 1]]
            seg_v = jv[jr[t]:jr[t + 1]]
            k = np.searchsorted(seg_c, i)
            assert seg_c[k] == i and seg_v.view(np.uint32)[k] == vals.view(np.uint32)[t]
    del rp_full


def test_offdiag_full(dev):
    import torch
    w = make("offdiag_f64")
    Ai, Aj, sr = w["A"], w["B"], w["semiring"]
    print(f"[full offdiag] m_i={Ai.nrows} m_j={Aj.nrows} nnz={Ai.nnz}+{Aj.nnz}", flush=True)
    O = sp.offdiag(upload(Ai, sr, dev), upload(Aj, sr, dev), sr)
    compare_full(O, oracle.offdiag(Ai, Aj, sr, threads=oracle.host_threads()), sr, "offdiag every row")
    ci, cj = col_counts(Ai), col_counts(Aj)
    assert sp.stats()["products"] == int((ci * cj).sum())
    # count semiring: sum of the block = sum_k c^i_k c^j_k
    K = sp.offdiag(upload(Ai, "count", dev), upload(Aj, "count", dev), "count")
    assert int(K.values[: K.nnz].to(torch.int64).sum().item()) == int((ci * cj).sum())
    check_lower(Ai, sr, dev, None, "offdiag diagonal block")


def test_offdiag_halves_full(dev):
    # Algorithm 3's half blocks at the off-diagonal workload's size, every row
    # of each half against the oracle's restriction of the whole block
    w = make("offdiag_f64")
    Ai, Aj, sr = w["A"], w["B"], w["semiring"]
    print(f"[full offdiag halves] m_i={Ai.nrows} m_j={Aj.nrows} nnz={Ai.nnz}+{Aj.nnz}", flush=True)
    top = sp.offdiag_half(upload(Ai, sr, dev), upload(Aj, sr, dev), "top", sr)
    right = sp.offdiag_half(upload(Ai, sr, dev), upload(Aj, sr, dev), "right", sr)
    ref = oracle.offdiag(Ai, Aj, sr, threads=oracle.host_threads())
    h = Ai.nrows // 2
    cut = int(ref.row_ptr[h])
    ref_top = oracle.Result(h, Aj.nrows, ref.row_ptr[:h + 1].copy(), ref.col_idx[:cut], ref.values[:cut],
                            ref.sum_abs[:cut])
    compare_full(top, ref_top, sr, "top half")
    keep = ref.col_idx >= Aj.nrows // 2
    rr = np.repeat(np.arange(Ai.nrows), np.diff(ref.row_ptr))
    rp = np.zeros(Ai.nrows + 1, dtype=np.int64)
    np.cumsum(np.bincount(rr[keep], minlength=Ai.nrows), out=rp[1:])
    ref_right = oracle.Result(Ai.nrows, Aj.nrows, rp, ref.col_idx[keep], ref.values[keep], ref.sum_abs[keep])
    compare_full(right, ref_right, sr, "right half")


@pytest.mark.parametrize("name", ["jaccard_large", "kmer_i32"])
def test_symm_full(dev, name):
    # Y = C x from the device's C_L at full size; sampled rows of Y against the
    # oracle's rows of the full product A A^T (the mirrored rows) times x
    import torch
    w = make(name)
    A, sr = w["A"], w["semiring"]
    print(f"[full symm {name}] m={A.nrows} nnz={A.nnz}", flush=True)
    C = sp.lower(upload(A, sr, dev), sr)
    xdt = np.float64 if sr in ("f64", "count") else np.float32
    rng = np.random.default_rng(5)
    x = rng.standard_normal(A.nrows).astype(xdt)
    y = sp.symm(C, torch.from_numpy(x).to(dev), sr).cpu().numpy().astype(np.float64)
    rows = sample_rows(A, 200, 23)
    Ain = A.with_values(A.values.astype(VDT[sr]) if VDT[sr] else None)
    R = oracle.offdiag(Ain, Ain, sr, rows=rows)
    rr = np.repeat(np.arange(len(rows)), np.diff(R.row_ptr))
    terms = R.values.astype(np.float64) * x.astype(np.float64)[R.col_idx]
    ref = np.bincount(rr, weights=terms, minlength=len(rows))
    scale = np.bincount(rr, weights=np.abs(terms), minlength=len(rows))
    tol = 1e-12 if sr in ("f64", "count") else 2.0 ** -24
    err = np.abs(y[rows] - ref)
    assert np.all(err <= tol * np.maximum(scale, np.abs(ref)) + 1e-300), float(err.max())


def test_accumulate_full_columns_split(dev):
    # jaccard_large's pattern as two stages (its columns split in half): the
    # overlap counts accumulated stage by stage equal the one-shot lower part
    # bit for bit
    import torch
    from paper_2608_09713_amd.workloads import CSR
    w = make("jaccard_large")
    A = w["A"]
    print(f"[full accumulate] m={A.nrows} nnz={A.nnz}", flush=True)
    half = A.ncols // 2
    rows = np.repeat(np.arange(A.nrows), np.diff(A.row_ptr))
    parts = []
    for lo, hi in ((0, half), (half, A.ncols)):
        sel = (A.col_idx >= lo) & (A.col_idx < hi)
        rp = np.zeros(A.nrows + 1, dtype=np.int64)
        np.cumsum(np.bincount(rows[sel], minlength=A.nrows), out=rp[1:])
        parts.append(CSR(A.nrows, hi - lo, rp, (A.col_idx[sel] - lo).astype(np.int32), None))
    full = sp.lower(upload(A, "count", dev), "count")
    first = sp.lower(upload(parts[0], "count", dev), "count")
    acc = sp.lower_accumulate(first, upload(parts[1], "count", dev), "count")
    del first
    assert acc.nnz == full.nnz
    assert torch.equal(acc.row_ptr, full.row_ptr)
    n = full.nnz
    assert torch.equal(acc.col_idx[:n], full.col_idx[:n])
    assert torch.equal(acc.values[:n], full.values[:n])


@pytest.mark.parametrize("name", ["jaccard_large", "offdiag_f64"])
def test_plan_execute_full(dev, name):
    # a plan at full size: an execution with new values equals the one-shot
    # product of those values bit for bit
    import torch
    w = make(name)
    A, sr = w["A"], w["semiring"]
    print(f"[full plan {name}] m={A.nrows} nnz={A.nnz}", flush=True)
    plan, C = sp.lower_plan(upload(A, sr, dev), sr)
    del C
    rng = np.random.default_rng(9)
    B = A.with_values(rng.random(A.nnz) + 0.5) if VDT[sr] else A
    Bd = upload(B, sr, dev)
    E = plan.execute(Bd.values)
    L = sp.lower(Bd, sr)
    assert E.nnz == L.nnz
    assert torch.equal(E.row_ptr, L.row_ptr)
    n = L.nnz
    assert torch.equal(E.col_idx[:n], L.col_idx[:n])
    assert torch.equal(E.values[:n].view(torch.uint8), L.values[:n].view(torch.uint8))
    plan.close()


def test_offdiag_self_full_wide_columns(dev):
    # offdiag(A, A) of jaccard_large's pattern (2^28 columns: dense column
    # starts of 1 GiB) is the full product: the mirror of the lower part,
    # counts bit for bit
    import torch
    w = make("jaccard_large")
    A = w["A"]
    print(f"[full offdiag(A, A)] m={A.nrows} n={A.ncols} nnz={A.nnz}", flush=True)
    Ad = upload(A, "count", dev)
    O = sp.offdiag(Ad, Ad, "count")
    M = sp.mirror(sp.lower(Ad, "count"), "count")
    assert O.nnz == M.nnz
    assert torch.equal(O.row_ptr, M.row_ptr)
    n = O.nnz
    assert torch.equal(O.col_idx[:n], M.col_idx[:n])
    assert torch.equal(O.values[:n], M.values[:n])
