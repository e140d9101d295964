"""Build the MCA HIP library (libmca.so) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmca.so")
SOURCES = ["mca_api.hip", "mlp_kernels.hip", "loop_kernel.hip", "slab_kernels.hip",
           "chain_kernels.hip", "channel_kernels.hip", "norm_kernels.hip",
           "tf_kernels.hip", "one_loop.hip"]

# Device code: gfx950 only; no fp contraction (explicit fmaf only, so the
# evaluation, commit and forward kernels round identically); packed fp32
# instructions disabled.
FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-shared",
         "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-result", "-I", os.path.join(ROOT, "include")]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the MCA library needs ROCm's hipcc")


def build(verbose: bool = False) -> str:
    """Compile libmca.so; returns its path.  Always recompiles."""
    tmp = LIB + ".tmp"
    cmd = [hipcc()] + FLAGS + ["-o", tmp] + [os.path.join(CSRC, s) for s in SOURCES]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if verbose or res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed building libmca.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
