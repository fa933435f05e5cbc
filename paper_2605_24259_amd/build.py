"""Build the gfx950 HIP library (librkc.so) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRCS = [os.path.join(PKG, "csrc", f) for f in ("rkc_replay.hip", "rkc_lean.hip")]
LIB = os.path.join(PKG, "librkc.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # packed FP32 instructions are kept off for all device code on this hardware
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # Leave regions whose branches are wave-uniform unstructured.  The per-pool event loops branch
    # only on wave-uniform values; structurizing those regions merged the outputs of two branches of
    # a refusal wrongly in some builds (a capacity refusal's b came out as the other branch's value),
    # which no build with this setting shows.
    "-mllvm", "-structurizecfg-skip-uniform-regions=true",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


# checking build: every readfirstlane also verifies that the active lanes agree (slower; used to
# run the GPU parity suite once against the uniformity assumptions of both kernels)
CHECK_LIB = os.path.join(PKG, "librkc_check.so")


def build(verbose: bool = False, check_uniform: bool = False) -> str:
    out = CHECK_LIB if check_uniform else LIB
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, *(["-DRKC_CHECK_UNIFORM"] if check_uniform else []), *SRCS, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    import sys
    print(build(verbose=True, check_uniform="--check-uniform" in sys.argv))
