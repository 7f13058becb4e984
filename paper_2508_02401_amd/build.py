"""Build libckv.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libckv.so")
SOURCES = [os.path.join(CSRC, n) for n in ("ckv_score.hip", "ckv_select.hip", "ckv_unit.hip", "ckv_decode.hip", "ckv_noalloc.hip", "ckv_api.cpp")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed fp32 instructions stay off: hipcc may otherwise form them from plain
# float code.
COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # MFMA results stay in VGPRs: the softmax reads them with VALU ops,
          # and accumulators in AGPRs would need a copy per element
          "-mllvm", "-amdgpu-mfma-vgpr-form",
          # kernel argument blocks indexed at run time (the multi-layer K
          # passes) are read in place; past InstCombine's default limit of
          # uses it copies such a block to per-lane scratch instead
          "-mllvm", "-instcombine-max-copied-from-constant-users=100000",
          "-I" + INCLUDE, "-I" + CSRC, "-Wall", "-Wno-unused-function"]


def build(verbose: bool = False) -> str:
    """Compile every source and link libckv.so. Returns the library path."""
    objs = []
    try:
        for src in SOURCES:
            obj = os.path.join(CSRC, os.path.basename(src) + ".o")
            lang = ["-x", "hip"]
            cmd = [HIPCC] + lang + COMMON + ["-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            objs.append(obj)
            subprocess.run(cmd, check=True)
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    finally:  # no stale objects, also when a compile fails
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
