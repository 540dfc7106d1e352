"""Randomised parity sweep: every entry point on many small seeded matrices
of varied shape, density and structure (empty rows, hub columns, dense rows,
one row, one column), each result checked against the oracle to the same bar
as the targeted tests."""
import dataclasses

import numpy as np
import pytest

import oracle
import paper_2608_09713_amd as sp
from paper_2608_09713_amd.workloads import CSR
from tests.parity import compare_full
from tests.test_gpu_parity import SEMIRINGS, VDT, _check_symm, _symm_ref, dev, upload  # noqa: F401

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1), (1, 50), (3, 2), (17, 300), (64, 64), (65, 1000), (200, 70000), (513, 900), (1500, 5000),
          (2100, 400)]


def _sweep_matrix(rng, m, n):
    lens = np.minimum(rng.poisson(rng.uniform(0, 12), size=m), n)
    lens[rng.random(m) < 0.15] = 0                       # empty rows
    dense = rng.random(m) < (0.02 if m > 50 else 0.0)   # a few dense rows
    lens[dense] = min(n, 400)
    hub = int(rng.integers(0, n)) if rng.random() < 0.5 else -1
    rows = []
    for i in range(m):
        c = set(rng.choice(n, size=int(lens[i]), replace=False).tolist()) if lens[i] else set()
        if hub >= 0 and rng.random() < 0.4:
            c.add(hub)
        rows.append(np.array(sorted(c), dtype=np.int32))
    rp = np.zeros(m + 1, dtype=np.int64)
    np.cumsum([len(r) for r in rows], out=rp[1:])
    ci = np.concatenate(rows) if rp[-1] else np.zeros(0, np.int32)
    return CSR(m, n, rp, ci, rng.standard_normal(len(ci)))


def _host(A, semiring):
    vdt = VDT[semiring]
    return A.with_values(A.values.astype(vdt) if vdt is not None else None)


@pytest.mark.parametrize("case", range(len(SHAPES) * 4))
def test_random_sweep(dev, case, monkeypatch):
    import torch
    rng = np.random.default_rng(1000 + case)
    m, n = SHAPES[case % len(SHAPES)]
    semiring = SEMIRINGS[case % len(SEMIRINGS)]
    A = _sweep_matrix(rng, m, n)
    B = _sweep_matrix(rng, int(rng.integers(1, 300)), n)
    print(f"[sweep {case}] {semiring} A {m}x{n} nnz={A.nnz}, B {B.nrows} rows nnz={B.nnz}", flush=True)
    Ad = upload(A, semiring, dev)
    L = oracle.lower(_host(A, semiring), semiring)
    C = sp.lower(Ad, semiring)
    compare_full(C, L, semiring, f"sweep {case} lower")
    compare_full(sp.offdiag(Ad, upload(B, semiring, dev), semiring),
                 oracle.offdiag(_host(A, semiring), _host(B, semiring), semiring), semiring, f"sweep {case} offdiag")
    for half in ("top", "right"):
        compare_full(sp.offdiag_half(upload(B, semiring, dev), Ad, half, semiring),
                     oracle.offdiag_half(_host(B, semiring), _host(A, semiring), half, semiring), semiring,
                     f"sweep {case} half {half}")
    # the mirror copies C_L's values: its bar is C_L's, the scale of each entry
    # (sum of |products|) mirrored with it
    Mr = oracle.mirror(m, L.row_ptr, L.col_idx, L.values)
    if L.sum_abs is not None:
        Mr = dataclasses.replace(Mr, sum_abs=oracle.mirror(m, L.row_ptr, L.col_idx, L.sum_abs).values)
    M = sp.mirror(C, semiring)
    compare_full(M, Mr, semiring, f"sweep {case} mirror")
    # and it is symmetric bit for bit: entry (i, j) holds the bits of (j, i)
    rp, ci, v = M.to_host()
    r = np.repeat(np.arange(m, dtype=np.int64), np.diff(rp))
    bits = v.view(np.uint32 if v.itemsize == 4 else np.uint64)
    o1, o2 = np.argsort(r * m + ci, kind="stable"), np.argsort(ci.astype(np.int64) * m + r, kind="stable")
    np.testing.assert_array_equal(bits[o1], bits[o2], err_msg=f"sweep {case}: mirror not symmetric")
    # the product with one column, buckets as chosen, forced and off
    xdt = np.float64 if semiring in ("f64", "count") else np.float32
    x = rng.standard_normal(m).astype(xdt)
    ref, scale = _symm_ref(L, x.astype(np.float64)[:, None])
    for b in (None, "1", "0"):
        if b is None:
            monkeypatch.delenv("SPSYRK_SYMM_BUCKETS", raising=False)
        else:
            monkeypatch.setenv("SPSYRK_SYMM_BUCKETS", b)
        y = sp.symm(C, torch.from_numpy(x).to(dev), semiring).cpu().numpy()
        _check_symm(y[:, None], ref, scale, semiring, f"sweep {case} symm buckets={b}")
    monkeypatch.delenv("SPSYRK_SYMM_BUCKETS", raising=False)
    # a second stage with other columns, accumulated
    if semiring != "jaccard":
        S = _sweep_matrix(rng, m, int(rng.integers(1, 2000)))
        compare_full(sp.lower_accumulate(C, upload(S, semiring, dev), semiring),
                     oracle.lower_accumulate(L, _host(S, semiring), semiring), semiring, f"sweep {case} accumulate")
    # a plan and an execution with new values
    plan, C0 = sp.lower_plan(Ad, semiring)
    compare_full(C0, L, semiring, f"sweep {case} plan")
    A2 = A.with_values(rng.standard_normal(A.nnz))
    E = plan.execute(upload(A2, semiring, dev).values)
    compare_full(E, oracle.lower(_host(A2, semiring), semiring), semiring, f"sweep {case} execute")
    plan.close()
