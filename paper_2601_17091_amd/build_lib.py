"""Build step: compile the HIP library in-tree for gfx950.

    python -m paper_2601_17091_amd.build_lib

produces ``paper_2601_17091_amd/librocket.so`` from ``csrc/``.  hipcc
cross-compiles the device code, so this runs on a machine without a GPU.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB = os.path.join(HERE, "librocket.so")
SOURCES = ["transform.hip", "plan.cpp", "generate.cpp", "minirocket.cpp"]
ARCH = "gfx950"


def hipcc() -> str:
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if os.path.exists(cand):
        return cand
    found = shutil.which("hipcc")
    if not found:
        raise RuntimeError("hipcc not found; the ROCm toolchain is required to build librocket.so")
    return found


def compile_flags() -> list[str]:
    return [
        "--offload-arch=" + ARCH,
        "-O3",
        "-std=c++17",
        "-fPIC",
        "-Wall",
        "-I", INCLUDE,
        # keep the compiler from forming packed fp32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # host arithmetic (the generator) exactly as written
        "-ffp-contract=off",
        # device code only: inputs are finite, so fmaxf is a plain v_max_f32
        # without NaN canonicalisation; host code (generator, planner,
        # MINIROCKET fit) keeps IEEE NaN semantics
        "-Xarch_device", "-fno-honor-nans",
        # MFMA results straight into VGPRs (no accumulator-register copies)
        "-mllvm", "-amdgpu-mfma-vgpr-form",
    ]


def build(verbose: bool = False) -> str:
    """Compile every source and link librocket.so (always rebuilds)."""
    os.makedirs(os.path.join(HERE, "_build"), exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(HERE, "_build", src + ".o")
        cmd = [hipcc()] + compile_flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True, stderr=subprocess.PIPE if not verbose else None)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
