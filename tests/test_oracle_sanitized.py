"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (host only).

Every entry point of the oracle library (lower, off-diagonal, half blocks, the
mirror, stage accumulation and the row-sharded driver on several threads) runs
on small seeded workloads of each shape, plus empty rows, an empty matrix and a
one-column matrix, in a child process whose sanitizer runtime aborts at the first
invalid access, leak aside (the interpreter's own allocations are not tracked).
The sanitized build must also give the same results as the ordinary one.  The
input generators are numpy code with no native part of their own.
"""
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = textwrap.dedent(r'''
    import sys
    import numpy as np
    sys.path.insert(0, sys.argv[2])
    import oracle
    from paper_2608_09713_amd import workloads as W

    san = oracle._load(sys.argv[1])
    plain = oracle._load()

    def rb(A, r0, r1):
        rp = A.row_ptr[r0:r1 + 1]
        v = None if A.values is None else A.values[rp[0]:rp[-1]]
        return W.CSR(r1 - r0, A.ncols, rp - rp[0], A.col_idx[rp[0]:rp[-1]], v)

    def same(a, b):
        assert np.array_equal(a.row_ptr, b.row_ptr) and np.array_equal(a.col_idx, b.col_idx)
        assert np.array_equal(a.values, b.values)

    cases = [
        (W.make("tiny_uniform_f64", scale_shift=3)["A"], "f64"),
        (W.make("kmer_i32", scale_shift=10)["A"], "count"),
        (W.make("jaccard_large", scale_shift=13)["A"], "jaccard"),
        (W.make("rmat20_f32", scale_shift=11)["A"], "f32"),
    ]
    # rows with nothing stored, a matrix with no rows, one column shared by all
    rp = np.array([0, 0, 2, 2, 3, 3], dtype=np.int64)
    E = W.CSR(5, 4, rp, np.array([1, 3, 1], dtype=np.int32), np.ones(3))
    Z = W.CSR(0, 4, np.zeros(1, dtype=np.int64), np.zeros(0, dtype=np.int32), np.zeros(0))
    O = W.CSR(6, 1, np.arange(7, dtype=np.int64), np.zeros(6, dtype=np.int32), np.arange(1.0, 7.0))
    for M in (E, Z, O):
        for sr in ("f64", "f32", "count", "jaccard"):
            cases.append((M, sr))
    for A, sr in cases:
        r = oracle.lower(A, sr, lib=san)
        same(r, oracle.lower(A, sr, lib=plain))
        same(oracle.lower(A, sr, lib=san, threads=4), r)
        h = A.nrows // 2
        Ai, Aj = rb(A, 0, h), rb(A, h, A.nrows)
        same(oracle.offdiag(Ai, Aj, sr, lib=san), oracle.offdiag(Ai, Aj, sr, lib=plain))
        for half in ("top", "right"):
            same(oracle.offdiag_half(Ai, Aj, half, sr, lib=san),
                 oracle.offdiag_half(Ai, Aj, half, sr, lib=plain))
        if sr != "jaccard":
            same(oracle.lower_accumulate(oracle.lower(Ai, sr, lib=san), Ai, sr, lib=san),
                 oracle.lower_accumulate(oracle.lower(Ai, sr, lib=plain), Ai, sr, lib=plain))
        if sr in ("f64", "f32", "count"):
            same(oracle.mirror(A.nrows, r.row_ptr, r.col_idx, r.values, lib=san),
                 oracle.mirror(A.nrows, r.row_ptr, r.col_idx, r.values, lib=plain))
    print("ok", len(cases))
''')


def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    asan_rt = subprocess.check_output(["g++", "-print-file-name=libasan.so"], text=True).strip()
    if not os.path.isabs(asan_rt):
        pytest.skip("no ASan runtime for g++")
    sys.path.insert(0, ROOT)
    import oracle
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    script = tmp_path / "child.py"
    script.write_text(CHILD)
    env = dict(os.environ, LD_PRELOAD=asan_rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    p = subprocess.run([sys.executable, str(script), lib, ROOT], env=env, cwd=str(tmp_path),
                       capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stdout[-3000:] + p.stderr[-6000:]
    assert p.stdout.strip().startswith("ok")
