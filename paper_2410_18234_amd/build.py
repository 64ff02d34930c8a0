"""Build the gfx950 HIP library libmdss.so in-tree (hipcc, no JIT cache)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libmdss.so")
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("api.hip", "induced.hip", "sample.hip", "tlp.hip", "optimum.hip", "alphabet.hip", "expsum.hip")]

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    # packed fp32 instructions are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no implicit contraction: every FMA in the kernels is written explicitly,
    # and the fp64 decisions of selection / acceptance round each operation
    "-ffp-contract=off",
    # matrix-core results go straight to VGPRs (no AGPR copies before the VALU reads them)
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-DMDSS_MFMA_MT=4", "-DMDSS_MFMA_NW=4",
    "-Wall",
]


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    out = LIB + ".tmp"
    cmd = [hipcc, *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-o", out, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libmdss.so")
    os.replace(out, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
