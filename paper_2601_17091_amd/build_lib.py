"""Build step: compile the HIP library in-tree for gfx950.

    python -m paper_2601_17091_amd.build_lib

produces ``paper_2601_17091_amd/librocket.so`` from ``csrc/`` (and the
checked build ``librocket_checked.so``, for debugging).  hipcc
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
CHECKED_LIB = os.path.join(HERE, "librocket_checked.so")
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
    """Compile every source and link librocket.so, and the checked build
    librocket_checked.so (transform.hip with ROCKET_CHECKED=1: device-side
    bounds checks for debugging); always rebuilds.  The compilations run in
    parallel."""
    os.makedirs(os.path.join(HERE, "_build"), exist_ok=True)
    jobs = []   # (command, object)
    objs = {False: [], True: []}
    for checked in (False, True):
        for src in SOURCES:
            if checked and src != "transform.hip":
                objs[True].append(os.path.join(HERE, "_build", src + ".o"))
                continue
            obj = os.path.join(HERE, "_build", src + (".checked.o" if checked else ".o"))
            cmd = [hipcc()] + compile_flags() + (["-DROCKET_CHECKED=1"] if checked else []) + \
                ["-c", os.path.join(CSRC, src), "-o", obj]
            jobs.append(cmd)
            objs[checked].append(obj)
    procs = []
    for cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stderr=None if verbose else subprocess.PIPE)))
    failed = []
    for cmd, pr in procs:
        _, err = pr.communicate()
        if pr.returncode != 0:
            failed.append((cmd, err))
    if failed:
        cmd, err = failed[0]
        raise RuntimeError("compilation failed: %s\n%s" % (" ".join(cmd), (err or b"").decode(errors="replace")))
    for checked, lib in ((False, LIB), (True, CHECKED_LIB)):
        tmp = lib + ".tmp%d" % os.getpid()
        cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs[checked]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
