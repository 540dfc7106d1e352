"""The C-ABI library builds, loads and exports every symbol of include/spsyrk.h;
host-side argument errors are reported without touching the GPU."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2608_09713_amd as sp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spsyrk.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(sp.LIB_PATH):
        from paper_2608_09713_amd import build
        build.build()
    return sp.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spsyrk_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("spsyrk_lower", "spsyrk_offdiag", "spsyrk_mirror", "spsyrk_status_string",
              "spsyrk_last_error_detail", "spsyrk_last_stats", "spsyrk_abi_version"):
        assert f in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.check_output(["nm", "-D", "--defined-only", sp.LIB_PATH]).decode()
    exported = set(re.findall(r"\bT (spsyrk_\w+)", out))
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    for f in declared_functions():
        getattr(lib, f)
    assert set(sp.EXPORTS) == set(declared_functions())


def test_status_strings_and_version(lib):
    assert lib.spsyrk_abi_version() == 2
    for code in range(8):
        assert lib.spsyrk_status_string(code)
    assert lib.spsyrk_status_string(99) == b"unknown status"


def _csr(nrows, ncols, nnz, rp=1, ci=1, v=None):
    return sp._Csr(nrows, ncols, nnz, rp, ci, v)


def _call_lower(lib, A, sr=0, out=True):
    o = sp._CsrOut()
    return lib.spsyrk_lower(ctypes.byref(A) if A is not None else None, sr, None, None,
                            ctypes.byref(o) if out else None)


def test_host_side_errors(lib):
    # none of these reach the device: the checks run before any allocation
    assert _call_lower(lib, None) == 1
    assert b"null" in lib.spsyrk_last_error_detail()
    assert _call_lower(lib, _csr(4, 4, 2, v=1), sr=7) == 1
    assert _call_lower(lib, _csr(-1, 4, 0)) == 1
    assert _call_lower(lib, _csr(1 << 31, 4, 0)) == 3
    assert _call_lower(lib, _csr(4, 1 << 31, 0)) == 3
    assert _call_lower(lib, _csr(4, 4, 1 << 31)) == 3
    assert _call_lower(lib, _csr(4, 4, 3, rp=None)) == 1
    assert _call_lower(lib, _csr(4, 4, 3, v=None), sr=0) == 1   # plus-times needs values
    assert _call_lower(lib, _csr(4, 4, 3, v=1), out=False) == 1
    a, b = _csr(4, 5, 1, v=1), _csr(4, 6, 1, v=1)
    o = sp._CsrOut()
    assert lib.spsyrk_offdiag(ctypes.byref(a), ctypes.byref(b), 0, None, None, ctypes.byref(o)) == 1
    assert b"columns" in lib.spsyrk_last_error_detail()
    c = _csr(4, 5, 1, v=1)
    assert lib.spsyrk_mirror(ctypes.byref(c), 0, None, None, ctypes.byref(o)) == 1
    assert b"square" in lib.spsyrk_last_error_detail()
    st = sp.Stats()
    assert lib.spsyrk_last_stats(ctypes.byref(st)) == 1  # no successful call yet on this thread


def test_host_side_errors_of_the_other_calls(lib):
    # the half blocks, the product from C_L, stage accumulation and plans
    # check their arguments before any device work
    o = sp._CsrOut()
    a, b = _csr(4, 5, 1, v=1), _csr(3, 5, 1, v=1)
    assert lib.spsyrk_offdiag_half(ctypes.byref(a), ctypes.byref(b), 2, 0, None, None, ctypes.byref(o)) == 1
    assert b"half" in lib.spsyrk_last_error_detail()
    b6 = _csr(3, 6, 1, v=1)
    assert lib.spsyrk_offdiag_half(ctypes.byref(a), ctypes.byref(b6), 0, 0, None, None, ctypes.byref(o)) == 1
    c = _csr(4, 4, 1, v=1)
    assert lib.spsyrk_symm(None, 0, 1, 1, 1, 1, 1, None, None) == 1
    assert lib.spsyrk_symm(ctypes.byref(_csr(4, 5, 1, v=1)), 0, 1, 1, 1, 1, 1, None, None) == 1
    assert b"square" in lib.spsyrk_last_error_detail()
    assert lib.spsyrk_symm(ctypes.byref(c), 0, 2, 1, 1, 1, 2, None, None) == 1   # ldx < k
    assert lib.spsyrk_symm(ctypes.byref(c), 0, -1, 1, 1, 1, 1, None, None) == 1  # k < 0
    assert lib.spsyrk_lower_accumulate(ctypes.byref(c), ctypes.byref(c), 3, None, None, ctypes.byref(o)) == 1
    assert b"Jaccard" in lib.spsyrk_last_error_detail()
    assert lib.spsyrk_lower_accumulate(ctypes.byref(c), ctypes.byref(_csr(5, 4, 1, v=1)), 0, None, None,
                                       ctypes.byref(o)) == 1
    assert lib.spsyrk_lower_execute(None, 1, None, None, ctypes.byref(o)) == 1
    assert lib.spsyrk_plan_destroy(None) == 0
    h = ctypes.c_void_p()
    assert lib.spsyrk_lower_plan(None, 0, None, None, ctypes.byref(h), ctypes.byref(o)) == 1
    assert not h.value
    assert lib.spsyrk_lower_plan(ctypes.byref(c), 0, None, None, None, ctypes.byref(o)) == 1


def test_noalloc_checks_before_device_work(lib):
    # argument errors and operands beyond the fixed scratch are refused on the
    # host, before the scratch or any device memory is touched
    c = _csr(4, 4, 1, v=1)
    assert lib.spsyrk_symm_noalloc(None, 0, 1, 1, 1, 1, 1, None) == 1
    assert lib.spsyrk_symm_noalloc(ctypes.byref(_csr(4, 5, 1, v=1)), 0, 1, 1, 1, 1, 1, None) == 1
    assert lib.spsyrk_symm_noalloc(ctypes.byref(c), 0, 2, 1, 1, 1, 2, None) == 1   # ldx < k
    big = _csr(1 << 21, 1 << 21, 0)
    assert lib.spsyrk_symm_noalloc(ctypes.byref(big), 0, 9, 1, 9, 1, 9, None) == 7
    assert b"scratch" in lib.spsyrk_last_error_detail()


def test_binding_refuses_to_run_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(sp, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(sp, "_lib", None)
    with pytest.raises(ImportError):
        sp.library()


def test_debug_build_exports_and_reports_itself(lib):
    """The build with the kernels' invariant checks exports the same symbols and
    says so; the ordinary build says it has none and reports no bits."""
    if not os.path.exists(sp.DEBUG_LIB_PATH):
        from paper_2608_09713_amd import build
        build.build(debug=True)
    out = subprocess.check_output(["nm", "-D", "--defined-only", sp.DEBUG_LIB_PATH]).decode()
    exported = set(re.findall(r"\bT (spsyrk_\w+)", out))
    assert not [f for f in declared_functions() if f not in exported]
    dbg = ctypes.CDLL(sp.DEBUG_LIB_PATH)
    assert dbg.spsyrk_debug_build() == 1
    assert lib.spsyrk_debug_build() == 0
    assert lib.spsyrk_debug_flags(None) == 1  # SPSYRK_ERR_INVALID_ARG, before any device call
