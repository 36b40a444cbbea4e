"""Builds libiefwd.so in-tree with hipcc for gfx950.

    python -m paper_2503_05130_amd.build      # or build() from Python

Every source is compiled on every call (the build check must really compile);
objects go to paper_2503_05130_amd/_build/ and the library to
paper_2503_05130_amd/libiefwd.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libiefwd.so")
ARCH = "gfx950"

SOURCES = ["gemm.hip", "attention.hip", "decode.hip", "layernorm.hip", "train.hip", "quota.cpp", "controller.cpp", "init_weights.cpp",
           "iefwd.cpp"]

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror",
    "-Wno-unused-command-line-argument",
    # no packed-FP32 (v_pk_*_f32) code generation
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in VGPRs: with the default heuristic the register
    # allocator splits them between AGPRs and VGPRs across the K loop's blocks
    # and copies every accumulator register with v_accvgpr_read/write on every
    # K step (48 copies per 24 MFMAs in the 128 x 96 tile)
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
# the init spec rounds every multiply and add separately
PER_FILE = {"init_weights.cpp": ["-ffp-contract=off"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, src + ".o")
    kind = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = [hipcc()] + COMMON + PER_FILE.get(src, []) + kind + ["-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def _check_stubs(lib: str) -> None:
    """Every kernel launched from host code must have its launch stub defined.

    clang's host pass can drop a kernel's stub without a diagnostic when the
    kernel body holds a device-only construct it cannot check on the host; the
    library would then fail to load at run time."""
    res = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True, check=True)
    missing = [line.split()[-1] for line in res.stdout.splitlines() if "__device_stub" in line]
    if missing:
        raise RuntimeError(f"undefined kernel launch stubs in {lib}: {missing[:4]}")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    _check_stubs(tmp)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
