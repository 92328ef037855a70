"""Build libstill.so (HIP, gfx950) in-tree with hipcc.

The library is four translation units compiled in parallel (the C ABI and
the consumer attention; the per-layer launch sequence for bf16 I/O; the same
for the fp32 validation mode; the backward pass) and linked into one shared
object."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libstill.so")
CSRC = os.path.join(PKG, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("still.hip", "layer_bf16.hip", "layer_fp32.hip", "backward.hip")]
HEADERS = [os.path.join(CSRC, f) for f in ("common.hpp", "gemm.hpp", "attn.hpp", "misc.hpp", "kproj.hpp",
                                           "consumer.hpp", "refine.hpp", "refine64.hpp", "host.hpp",
                                           "layer.hpp", "bwd.hpp")] + [os.path.join(ROOT, "include", "still.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         # keep hipcc from forming packed fp32 (v_pk_*_f32) instructions
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         # MFMA operands/results in VGPRs; AGPRs then serve as fast spill space
         "-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def _filter(stderr: str) -> str:
    return "\n".join(l for l in stderr.splitlines() if "packed-fp32-ops" not in l)


def build_library(verbose: bool = False) -> str:
    """Compile the HIP library; always recompiles. Returns the library path."""
    objs = [os.path.join(CSRC, os.path.basename(src) + ".o") for src in SOURCES]
    procs = []
    for src, obj in zip(SOURCES, objs):
        cmd = [HIPCC, *FLAGS, "-c", "-o", obj, src]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
    errors = []
    for src, p in zip(SOURCES, procs):
        out, err = p.communicate()
        err = _filter(err)
        if p.returncode != 0:
            errors.append(f"{os.path.basename(src)}: hipcc failed ({p.returncode}):\n{err}")
        elif verbose and err.strip():
            print(err, file=sys.stderr)
    if errors:
        raise RuntimeError("\n".join(errors))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed ({r.returncode}):\n{_filter(r.stderr)}")
    os.replace(tmp, LIB)
    for obj in objs:
        os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
