"""Error paths of the C-ABI on the GPU: an allocator that fails at its k-th
allocation, for every k a call makes, must give SPSYRK_ERR_OOM, a zeroed
output struct and no live allocation; the NULL allocator (stream-ordered HIP
allocations) must work for plans, executions and their release.

Inputs are small seeded matrices that take both row classes (a hub column
makes heavy rows), so that every allocation site of a call is reached.
"""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2608_09713_amd as sp
from paper_2608_09713_amd.workloads import CSR
from tests.helpers import random_csr
from tests.parity import compare_full

pytestmark = pytest.mark.gpu

OOM = 4


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available()
    sp.library()
    return "cuda:0"


class CountingAllocator:
    """Device allocator backed by torch; the allocation numbered ``fail_at``
    (0-based) returns NULL.  ``live`` maps pointers to tensors not yet freed."""

    def __init__(self, device, fail_at=None):
        import torch
        self.torch = torch
        self.device = device
        self.fail_at = fail_at
        self.count = 0
        self.live = {}
        self._a = sp._ALLOC(self._alloc)
        self._f = sp._FREE(self._free)
        self.struct = sp._Allocator(self._a, self._f, None)

    def _alloc(self, ctx, nbytes):
        k = self.count
        self.count += 1
        if self.fail_at is not None and k == self.fail_at:
            return None
        t = self.torch.empty(int(nbytes), dtype=self.torch.uint8, device=self.device)
        self.live[t.data_ptr()] = t
        return t.data_ptr()

    def _free(self, ctx, p):
        self.live.pop(p, None)


def _hub_matrix(seed, m=700, n=900, dtype=np.float64):
    # random rows plus one column shared by every third row: heavy rows by products
    rng = np.random.default_rng(seed)
    A = random_csr(rng, m, n, 0.01, dtype=dtype, signed=False)
    D = np.zeros((m, n))
    P = np.zeros((m, n), dtype=bool)
    rows = np.repeat(np.arange(m), np.diff(A.row_ptr))
    D[rows, A.col_idx] = A.values
    P[rows, A.col_idx] = True
    P[::3, 5] = True
    D[::3, 5] = 1.5
    r, c = np.nonzero(P)
    rp = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(np.bincount(r, minlength=m), out=rp[1:])
    return CSR(m, n, rp, c.astype(np.int32), D[r, c].astype(dtype))


def _dev_csr(A, dev):
    return sp.DeviceCSR.from_host(A, dev)


def _struct(C, with_values=True):
    return sp._Csr(C.nrows, C.ncols, C.nnz, C.row_ptr.data_ptr(), C.col_idx.data_ptr(),
                   C.values.data_ptr() if (with_values and C.values is not None) else None)


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _zeroed(out):
    return all(getattr(out, f) in (0, None) for f, _ in out._fields_)


def _sweep(dev, invoke, what):
    """invoke(alloc, out) -> rc.  Count the allocations of a good call, then
    fail each one in turn."""
    import torch
    good = CountingAllocator(dev)
    out = sp._CsrOut()
    rc = invoke(good, out)
    assert rc == 0, f"{what}: {sp.library().spsyrk_last_error_detail()}"
    n = good.count
    assert n > 0
    print(f"[oom sweep] {what}: {n} allocations", flush=True)
    for k in range(n):
        al = CountingAllocator(dev, fail_at=k)
        out = sp._CsrOut()
        rc = invoke(al, out)
        torch.cuda.synchronize()
        assert rc == OOM, f"{what}: allocation {k} of {n} failed but the call returned {rc}"
        assert _zeroed(out), f"{what}: output not zeroed after failing allocation {k}"
        assert not al.live, f"{what}: {len(al.live)} allocations left live after failing allocation {k}"
        assert al.count == k + 1, f"{what}: allocated again after the failure at {k}"
    return n


@pytest.mark.parametrize("semiring", ["f64", "jaccard"])
def test_oom_at_every_allocation_lower_offdiag_mirror(dev, semiring):
    lib = sp.library()
    sr = sp.SEMIRINGS[semiring]
    A = _hub_matrix(1)
    B = _hub_matrix(2, m=500)
    if semiring == "jaccard":
        A, B = A.with_values(None), B.with_values(None)
    dA, dB = _dev_csr(A, dev), _dev_csr(B, dev)
    a, b = _struct(dA), _struct(dB)
    s = _stream()
    _sweep(dev, lambda al, o: lib.spsyrk_lower(ctypes.byref(a), sr, ctypes.byref(al.struct), s, ctypes.byref(o)),
           f"lower {semiring}")
    _sweep(dev, lambda al, o: lib.spsyrk_offdiag(ctypes.byref(a), ctypes.byref(b), sr, ctypes.byref(al.struct), s,
                                                 ctypes.byref(o)), f"offdiag {semiring}")
    for half in (0, 1):
        _sweep(dev, lambda al, o: lib.spsyrk_offdiag_half(ctypes.byref(a), ctypes.byref(b), half, sr,
                                                          ctypes.byref(al.struct), s, ctypes.byref(o)),
               f"offdiag_half {half} {semiring}")
    C = sp.lower(dA, semiring)
    c = _struct(C)
    _sweep(dev, lambda al, o: lib.spsyrk_mirror(ctypes.byref(c), sr, ctypes.byref(al.struct), s, ctypes.byref(o)),
           f"mirror {semiring}")


def test_oom_at_every_allocation_mirror_slabs(dev, monkeypatch):
    # the slab planner's histograms and per-slab buffers
    monkeypatch.setenv("SPSYRK_MIRROR_SLAB", "500")
    lib = sp.library()
    C = sp.lower(_dev_csr(_hub_matrix(3), dev), "f64")
    c = _struct(C)
    s = _stream()
    _sweep(dev, lambda al, o: lib.spsyrk_mirror(ctypes.byref(c), 0, ctypes.byref(al.struct), s, ctypes.byref(o)),
           "mirror in slabs")


def test_oom_at_every_allocation_two_pass(dev, monkeypatch):
    monkeypatch.setenv("SPSYRK_TWO_PASS", "1")
    lib = sp.library()
    dA, dB = _dev_csr(_hub_matrix(4), dev), _dev_csr(_hub_matrix(5, m=300), dev)  # kept alive
    a, b = _struct(dA), _struct(dB)
    s = _stream()
    _sweep(dev, lambda al, o: lib.spsyrk_lower(ctypes.byref(a), 0, ctypes.byref(al.struct), s, ctypes.byref(o)),
           "lower two-pass")
    _sweep(dev, lambda al, o: lib.spsyrk_offdiag(ctypes.byref(a), ctypes.byref(b), 0, ctypes.byref(al.struct), s,
                                                 ctypes.byref(o)), "offdiag two-pass")


@pytest.mark.parametrize("buckets,split", [("0", "0"), ("12", "0"), ("0", "1")])
def test_oom_at_every_allocation_symm(dev, buckets, split, monkeypatch):
    import torch
    monkeypatch.setenv("SPSYRK_SYMM_BUCKETS", buckets)
    monkeypatch.setenv("SPSYRK_SYMM_SPLIT", split)
    lib = sp.library()
    C = sp.lower(_dev_csr(_hub_matrix(6), dev), "f64")
    c = _struct(C)
    X = torch.rand(C.nrows, 1, dtype=torch.float64, device=dev)
    Y = torch.empty_like(X)
    s = _stream()

    def call(al, o):
        return lib.spsyrk_symm(ctypes.byref(c), 0, 1, ctypes.c_void_p(X.data_ptr()), 1,
                               ctypes.c_void_p(Y.data_ptr()), 1, ctypes.byref(al.struct), s)
    _sweep(dev, call, f"symm buckets={buckets} split={split}")


@pytest.mark.parametrize("semiring", ["f64", "count"])
def test_oom_at_every_allocation_accumulate(dev, semiring):
    lib = sp.library()
    sr = sp.SEMIRINGS[semiring]
    A1, A2 = _hub_matrix(7), _hub_matrix(8)
    if semiring == "count":
        A1, A2 = A1.with_values(None), A2.with_values(None)
    P = sp.lower(_dev_csr(A1, dev), semiring)
    p = _struct(P)
    dA = _dev_csr(A2, dev)  # kept alive for the calls
    a = _struct(dA)
    s = _stream()
    _sweep(dev, lambda al, o: lib.spsyrk_lower_accumulate(ctypes.byref(p), ctypes.byref(a), sr,
                                                          ctypes.byref(al.struct), s, ctypes.byref(o)),
           f"accumulate {semiring}")


def test_oom_at_every_allocation_plan_and_execute(dev):
    import torch
    lib = sp.library()
    A = _hub_matrix(9)
    dA = _dev_csr(A, dev)  # kept alive for the calls
    a = _struct(dA)
    s = _stream()
    handles = []

    def plan(al, o):
        h = ctypes.c_void_p()
        rc = lib.spsyrk_lower_plan(ctypes.byref(a), 0, ctypes.byref(al.struct), s, ctypes.byref(h), ctypes.byref(o))
        if rc == 0:
            handles.append((h, al, {o.row_ptr, o.col_idx, o.values}))
        else:
            assert not h.value, "a failed plan call handed out a plan"
        return rc
    _sweep(dev, plan, "lower_plan")
    h, al_plan, c_arrays = handles[0]
    vals = torch.from_numpy(A.values * 2.0).to(dev)
    _sweep(dev, lambda al, o: lib.spsyrk_lower_execute(h, ctypes.c_void_p(vals.data_ptr()), ctypes.byref(al.struct),
                                                       s, ctypes.byref(o)), "lower_execute")
    assert lib.spsyrk_plan_destroy(h) == 0
    # what stays is C_L itself (the caller's); every plan buffer was released
    assert set(al_plan.live) == c_arrays, "plan buffers left after spsyrk_plan_destroy"


def _hip():
    # the HIP runtime already loaded by torch and the library (same soname,
    # so the loader hands back that copy)
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    hip.hipFreeAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    return hip


def _take(out, dtype, stream):
    """Copy a result allocated with the NULL allocator (hipMallocAsync on the
    call's stream) to the host, then return it with hipFreeAsync."""
    import torch
    rp = np.empty(out.nrows + 1, dtype=np.int64)
    ci = np.empty(out.nnz, dtype=np.int32)
    v = np.empty(out.nnz, dtype=dtype)
    hip = _hip()
    torch.cuda.synchronize()
    assert hip.hipMemcpy(rp.ctypes.data, out.row_ptr, rp.nbytes, 2) == 0  # device to host
    if out.nnz:
        assert hip.hipMemcpy(ci.ctypes.data, out.col_idx, ci.nbytes, 2) == 0
        assert hip.hipMemcpy(v.ctypes.data, out.values, v.nbytes, 2) == 0
    for p in (out.row_ptr, out.col_idx, out.values):
        if p:
            assert hip.hipFreeAsync(p, stream) == 0
    assert hip.hipStreamSynchronize(stream) == 0
    return rp, ci, v


def test_null_allocator_lower_and_plan(dev):
    # the NULL allocator takes stream-ordered HIP allocations: results are the
    # same, and a plan made with it executes and is released by destroy
    import torch
    lib = sp.library()
    A = _hub_matrix(10)
    dA = _dev_csr(A, dev)  # kept alive for the calls
    a = _struct(dA)
    s = _stream()
    ref = oracle.lower(A, "f64")
    out = sp._CsrOut()
    assert lib.spsyrk_lower(ctypes.byref(a), 0, None, s, ctypes.byref(out)) == 0
    rp, ci, v = _take(out, np.float64, s)
    np.testing.assert_array_equal(rp, ref.row_ptr)
    np.testing.assert_array_equal(ci, ref.col_idx)
    np.testing.assert_allclose(v, ref.values, rtol=1e-12)
    h = ctypes.c_void_p()
    out = sp._CsrOut()
    assert lib.spsyrk_lower_plan(ctypes.byref(a), 0, None, s, ctypes.byref(h), ctypes.byref(out)) == 0
    assert h.value
    _take(out, np.float64, s)
    vals = torch.from_numpy(A.values * 3.0).to(dev)
    ref3 = oracle.lower(A.with_values(A.values * 3.0), "f64")
    for _ in range(2):
        out = sp._CsrOut()
        assert lib.spsyrk_lower_execute(h, ctypes.c_void_p(vals.data_ptr()), None, s, ctypes.byref(out)) == 0
        rp, ci, v = _take(out, np.float64, s)
        np.testing.assert_array_equal(ci, ref3.col_idx)
        np.testing.assert_allclose(v, ref3.values, rtol=1e-12)
    assert lib.spsyrk_plan_destroy(h) == 0
    torch.cuda.synchronize()
