"""Build libctcbeam.so (C ABI + gfx950 kernels) in-tree with hipcc.

Usage: python -m paper_2508_07315_amd.build_lib [--phase-clocks]

--phase-clocks builds the profiling flavour libctcbeam_phase.so instead: the
same library with per-phase cycle counters in the decode kernel
(CTCBEAM_PHASE_CLOCKS; read by ``paper_2508_07315_amd.phase_profile``).  The
product library is never built with them.
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
LIB_PHASE = os.path.join(PKG, "libctcbeam_phase.so")
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


KERNEL_UNITS = ["ctcbeam_kernel_lpt1.hip", "ctcbeam_kernel_lpt2.hip", "ctcbeam_kernel_lpt4.hip",
                "ctcbeam_kernel_lpt8.hip", "ctcbeam_kernel_lpt1_rep.hip", "ctcbeam_kernel_lpt2_rep.hip",
                "ctcbeam_kernel_lpt4_rep.hip", "ctcbeam_kernel_lpt8_rep.hip", "ctcbeam_greedy_v256.hip", "ctcbeam_greedy_v1024.hip",
                "ctcbeam_greedy_v4096.hip", "ctcbeam_workspace.hip",
                "ctcbeam_noalloc.hip", "ctcbeam_small.hip"]


def build(verbose: bool = False, jobs: int = 0, phase_clocks: bool = False) -> str:
    from concurrent.futures import ThreadPoolExecutor
    jobs = jobs or max(1, min(len(KERNEL_UNITS) + 1, os.cpu_count() or 1))
    lib = LIB_PHASE if phase_clocks else LIB
    extra = ["-DCTCBEAM_PHASE_CLOCKS"] if phase_clocks else []
    with tempfile.TemporaryDirectory(prefix="ctcbeam_build_") as tmp:
        cmds, objs = [], []
        for unit in KERNEL_UNITS:
            o = os.path.join(tmp, unit.replace(".hip", ".o"))
            cmds.append(["hipcc", *COMMON, *extra, *DEVICE, "-c", os.path.join(CSRC, unit), "-o", o])
            objs.append(o)
        h_o = os.path.join(tmp, "host.o")
        cmds.append(["hipcc", *COMMON, "-c", os.path.join(CSRC, "ctcbeam_host.cpp"), "-o", h_o])
        objs.append(h_o)
        with ThreadPoolExecutor(jobs) as ex:
            list(ex.map(_run, cmds))
        out_tmp = lib + f".tmp{os.getpid()}"
        _run(["hipcc", *DEVICE, "-shared", "-fPIC", *objs, "-o", out_tmp])
        os.replace(out_tmp, lib)
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    build(verbose=True, phase_clocks="--phase-clocks" in sys.argv[1:])
