"""The debug build (kernels compiled with their invariant checks) on the GPU.

A child process loads libspsyrk_debug.so (SPSYRK_DEBUG=1), runs the lower
product on light-only, heavy-row and power-law inputs in every semiring, the
mirror and the off-diagonal block, compares each result with the oracle, and
checks after every call that no kernel raised a check bit.  A raised bit would
mean an output slot written outside its row or a numeric pass that disagrees
with its symbolic count, which element-wise parity at these sizes could miss if
the stray write landed where nothing is compared.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent(r'''
    import sys
    import numpy as np
    sys.path.insert(0, sys.argv[1])
    import oracle
    import paper_2608_09713_amd as sp
    from paper_2608_09713_amd import workloads as W
    from tests.helpers import csr_from_dense
    from tests.parity import compare_full

    import torch
    assert torch.cuda.is_available()
    assert sp.debug_build(), "SPSYRK_DEBUG=1 did not load the debug build"
    dev = "cuda:0"

    def check(what):
        f = sp.debug_flags()
        assert f == 0, "%s: debug check bits %#x" % (what, f)
        print("ok", what, flush=True)

    D = np.zeros((2500, 4))
    D[:, 2] = 1.0
    D[::3, 0] = 0.5
    heavy = csr_from_dense(D)
    cases = [(W.make("tiny_uniform_f64")["A"], "f64", "tiny uniform"),
             (W.make("kmer_i32", scale_shift=6)["A"], "count", "kmer 2^14 rows"),
             (W.make("jaccard_large", scale_shift=9)["A"], "jaccard", "jaccard 2^14 rows"),
             (W.make("rmat20_f32", scale_shift=6)["A"], "f32", "rmat scale 14")]
    dense = {"f64": heavy, "f32": csr_from_dense(D, dtype=np.float32),
             "count": heavy.with_values(None), "jaccard": heavy.with_values(None)}
    cases += [(dense[sr], sr, "dense column " + sr) for sr in ("f64", "f32", "count", "jaccard")]
    for A, sr, what in cases:
        C = sp.lower(sp.DeviceCSR.from_host(A, dev), sr)
        check(what)
        if what.startswith("dense column"):
            assert sp.stats()["heavy_rows"] > 0
        ref = oracle.lower(A, sr)
        compare_full(C, ref, sr, what)
        if sr in ("f64", "f32") and what.startswith("rmat"):
            F = sp.mirror(C, sr)
            check(what + " mirror")
            compare_full(F, oracle.mirror(A.nrows, ref.row_ptr, ref.col_idx, ref.values), sr, what + " mirror")
    X = W.make("offdiag_f64", scale_shift=6)
    Ai, Aj = sp.DeviceCSR.from_host(X["A"], dev), sp.DeviceCSR.from_host(X["B"], dev)
    compare_full(sp.offdiag(Ai, Aj, "f64"), oracle.offdiag(X["A"], X["B"], "f64"), "f64", "offdiag 2^13 rows")
    check("offdiag 2^13 rows")
    print("done", flush=True)
''')


@pytest.mark.gpu
def test_debug_build_raises_no_check(tmp_path):
    lib = os.path.join(ROOT, "paper_2608_09713_amd", "libspsyrk_debug.so")
    if not os.path.exists(lib):
        pytest.fail("libspsyrk_debug.so is missing: run __graft_entry__.build() first")
    script = tmp_path / "child.py"
    script.write_text(CHILD)
    env = dict(os.environ, SPSYRK_DEBUG="1")
    p = subprocess.run([sys.executable, "-u", str(script), ROOT], env=env, cwd=ROOT,
                       capture_output=True, text=True, timeout=240)
    assert p.returncode == 0, p.stdout[-3000:] + p.stderr[-4000:]
    assert "done" in p.stdout
