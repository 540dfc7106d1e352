"""Host-side logic of the library checked on the CPU (no GPU, no HIP runtime):
plain C++ headers of the library compiled with g++ into small check programs."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2608_09713_amd", "csrc")


def _run_check(name, tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = tmp_path / name
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-Wall", "-Werror", "-I", CSRC,
                           os.path.join(HERE, "host", name + ".cpp"), "-o", str(exe)])
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    return out.stdout


def test_symm_bucket_layout_fits_lds_tables(tmp_path):
    # every forced bucket size at every row count up to 2^24 keeps the number
    # of buckets within the kernels' LDS tables
    assert _run_check("symm_layout_check", tmp_path).startswith("ok")
