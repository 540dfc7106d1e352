"""Build libspsyrk.so (hipcc, gfx950) in-tree.

Usage: python -m paper_2608_09713_amd.build
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libspsyrk.so")
# the same sources with the kernels' invariant checks compiled in (SPSYRK_DEBUG)
DEBUG_LIB = os.path.join(PKG, "libspsyrk_debug.so")
ARCH = os.environ.get("SPSYRK_OFFLOAD_ARCH", "gfx950")

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # packed fp32 instructions are kept out of the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(verbose: bool = False, debug: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    flags = FLAGS + (["-DSPSYRK_DEBUG=1"] if debug else [])
    target = DEBUG_LIB if debug else LIB
    objs = []
    tmpdir = os.path.join(PKG, "_build", "debug") if debug else os.path.join(PKG, "_build")
    os.makedirs(tmpdir, exist_ok=True)
    procs = []
    for src in sources():
        obj = os.path.join(tmpdir, os.path.basename(src) + ".o")
        cmd = [hipcc, *[f for f in flags if f != "-shared"], "-c", src, "-o", obj]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        for src, text in failed:
            sys.stderr.write(f"--- {src}\n{text}\n")
        raise RuntimeError("hipcc failed for " + ", ".join(os.path.basename(s) for s, _ in failed))
    tmp = target + f".tmp{os.getpid()}"
    subprocess.check_call([hipcc, *flags, *objs, "-o", tmp])
    os.replace(tmp, target)
    return target


if __name__ == "__main__":
    print(build(verbose=True))
