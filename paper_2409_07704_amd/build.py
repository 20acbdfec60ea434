"""Compile libmas (the HIP kernels and the C-ABI host code) for gfx950.

Builds in-tree: ``paper_2409_07704_amd/libmas.so``.  hipcc cross-compiles
without a GPU.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmas.so")
TRACE_LIB = os.path.join(PKG, "libmas_trace.so")
SOURCES = ["mas_kernels.hip", "mas_text.hip", "mas_loglik.hip", "mas_api.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # bit-exact fp32: no contraction, IEEE denormals on the device
    "-ffp-contract=off",
    "-fno-gpu-flush-denormals-to-zero",
    # keep the compiler from emitting packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


# The product library, and the debug build that records a timeline of each
# launch (MAS_TRACE: wall-clock stamps of every wave's milestones, see trace.py).
VARIANTS = {LIB: [], TRACE_LIB: ["-DMAS_TRACE"]}


def _noise_free(stderr: str) -> str:
    # hipcc's host pass does not know the packed-fp32 feature; that warning is harmless.
    noise = "'-packed-fp32-ops' is not a recognized feature for this target (ignoring feature)"
    return "\n".join(l for l in stderr.splitlines()
                     if noise not in l and "warning generated" not in l and "warnings generated" not in l)


def build(verbose: bool = False) -> str:
    """Compile every source into libmas.so and libmas_trace.so (always
    recompiles; the two builds run in parallel)."""
    procs = {}
    for out, extra in VARIANTS.items():
        cmd = [HIPCC, *FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, *[os.path.join(CSRC, s) for s in SOURCES],
               "-o", out + ".tmp"]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs[out] = subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)
    errors = []
    for out, pr in procs.items():
        _, stderr = pr.communicate()
        err = _noise_free(stderr)
        if pr.returncode != 0:
            errors.append(f"hipcc failed for {os.path.basename(out)} ({pr.returncode}):\n{err}")
        elif err.strip():
            # Any other diagnostic (an inline-assembly constraint the compiler
            # cannot honour, say) fails the build.
            errors.append(f"hipcc reported warnings for {os.path.basename(out)}:\n{err}")
    if errors:
        for out in procs:
            if os.path.exists(out + ".tmp"):
                os.remove(out + ".tmp")
        raise RuntimeError("\n".join(errors))
    for out in procs:
        os.replace(out + ".tmp", out)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
