"""Build libstill.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libstill.so")
SOURCES = [os.path.join(PKG, "csrc", "still.hip")]
HEADERS = [os.path.join(PKG, "csrc", f) for f in ("common.hpp", "gemm.hpp", "attn.hpp", "misc.hpp", "kproj.hpp", "consumer.hpp", "refine.hpp")] + \
          [os.path.join(ROOT, "include", "still.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         # keep hipcc from forming packed fp32 (v_pk_*_f32) instructions
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         # MFMA operands/results in VGPRs; AGPRs then serve as fast spill space
         "-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def build_library(verbose: bool = False) -> str:
    """Compile the HIP library; always recompiles. Returns the library path."""
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
