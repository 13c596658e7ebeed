"""Build libctcbeam.so (C ABI + gfx950 kernels) in-tree with hipcc.

Usage: python -m paper_2508_07315_amd.build_lib
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libctcbeam.so")
ARCH = os.environ.get("CTCBEAM_ARCH", "gfx950")

# -ffp-contract=off: the fp32 score fold must not be fused into FMAs (the
# token outputs are compared bit for bit with the oracle's fp32 fold).
# -packed-fp32-ops off: no v_pk_*_f32 generated from scalar float code.
COMMON = ["-O3", "-fPIC", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
          f"-I{os.path.join(ROOT, 'include')}"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("command failed: " + " ".join(cmd))


def build(verbose: bool = False) -> str:
    with tempfile.TemporaryDirectory(prefix="ctcbeam_build_") as tmp:
        k_o = os.path.join(tmp, "kernel.o")
        h_o = os.path.join(tmp, "host.o")
        _run(["hipcc", *COMMON, *DEVICE, "-c", os.path.join(CSRC, "ctcbeam_kernel.hip"), "-o", k_o])
        _run(["hipcc", *COMMON, "-c", os.path.join(CSRC, "ctcbeam_host.cpp"), "-o", h_o])
        out_tmp = LIB + f".tmp{os.getpid()}"
        _run(["hipcc", *DEVICE, "-shared", "-fPIC", k_o, h_o, "-o", out_tmp])
        os.replace(out_tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
