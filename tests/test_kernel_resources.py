"""Register and occupancy budgets of the hot kernels, read from the compiler's
resource report for gfx950 (no GPU needed).

The heavy-row numeric pass keeps three workgroups of 512 threads on a compute
unit (its LDS allows three), which takes six wavefronts per SIMD, so at most
80 VGPRs; at 88 only two workgroups fit and the pass runs about 40% longer.
The symbolic pass keeps eight wavefronts per SIMD (64 VGPRs).  The light-row
kernel keeps three wavefronts per SIMD for the plus-times semirings, at the
price of a spill of a few words per lane (at two wavefronts per SIMD it needs
175 VGPRs and no spill, and measures slower); the count and Jaccard kernels
fit without one.  No other kernel here may spill.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2608_09713_amd import build

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _report(src):
    flags = [f for f in build.FLAGS if f not in ("-shared",)]
    cmd = [HIPCC, *flags, "--cuda-device-only", "-c", "-Rpass-analysis=kernel-resource-usage",
           os.path.join(build.CSRC, src), "-o", os.devnull]
    out = subprocess.run(cmd, capture_output=True, text=True, check=True).stderr
    kernels = {}
    name = None
    for line in out.splitlines():
        m = re.search(r"remark:\s+Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            kernels[name] = {}
            continue
        m = re.search(r"remark:\s+(VGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]|LDS Size \[bytes/block\]): "
                      r"(\d+)", line)
        if m and name:
            kernels[name][m.group(1).split()[0] if not m.group(1).startswith("LDS") else "LDS"] = int(m.group(2))
    return kernels


pytestmark = pytest.mark.skipif(shutil.which(HIPCC) is None and not os.path.exists(HIPCC),
                                reason="hipcc not available")


def test_heavy_kernel_budgets():
    ks = {k: v for k, v in _report("heavy.hip").items() if "heavy_kernel" in k}
    assert len(ks) == 16  # four semirings x symbolic/numeric x lower/off-diagonal
    for name, r in ks.items():
        numeric = re.search(r"heavy_kernelILi\dELb1E", name) is not None
        assert r["ScratchSize"] == 0, name
        if numeric:  # three workgroups of eight wavefronts per compute unit (160 KiB of LDS)
            assert r["VGPRs"] <= 80 and r["Occupancy"] >= 6 and 3 * r["LDS"] <= 160 * 1024, (name, r)
        else:  # four
            assert r["VGPRs"] <= 64 and r["Occupancy"] >= 8 and 4 * r["LDS"] <= 160 * 1024, (name, r)


def test_light_kernel_budgets():
    ks = {k: v for k, v in _report("light_fused.hip").items() if "fused_kernel" in k}
    assert len(ks) == 8
    for name, r in ks.items():
        if re.search(r"fused_kernelILi[01]E", name):  # plus-times in f64 and f32
            assert r["Occupancy"] >= 3 and r["ScratchSize"] <= 40, (name, r)
        else:
            assert r["Occupancy"] >= 3 and r["ScratchSize"] == 0, (name, r)


def test_local_sort_budgets():
    # the packed column sort's first launch holds groups of up to 2048
    # records: at most 18 KiB of LDS and 72 VGPRs, so that seven workgroups
    # of four wavefronts share a compute unit (the second launch, for the
    # rare larger groups, keeps the 4096-record LDS arrays); no spills
    ks = _report("radix.hip")
    small = {k: v for k, v in ks.items() if "local_sort_packILi" in k}
    big = {k: v for k, v in ks.items() if "local_sort_pack_bigILi" in k}
    # f64, f32, count and Jaccard records, and f64 and f32 records that carry
    # the values in place of the entry indices
    assert len(small) == 6 and len(big) == 6
    for name, r in small.items():
        assert r["ScratchSize"] == 0 and r["VGPRs"] <= 72 and r["LDS"] <= 18 * 1024, (name, r)
        assert r["Occupancy"] >= 7 and 7 * r["LDS"] <= 160 * 1024, (name, r)
    for name, r in big.items():
        assert r["ScratchSize"] == 0 and r["LDS"] <= 36 * 1024, (name, r)
