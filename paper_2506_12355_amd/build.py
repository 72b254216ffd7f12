"""Build the gfx950 attention library in place: ``libqm_attn.so`` beside this file.

Usage: ``python -m paper_2506_12355_amd.build`` (or call :func:`build`).  It
always recompiles.  hipcc cross-compiles for gfx950 without a GPU present.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libqm_attn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)

SOURCES = ["qm_attn.cpp", "attn_fwd_gfx950.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # device code never sees a NaN in valid use: fmax needs no quieting of its inputs
    "-Xarch_device", "-fno-honor-nans",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = shutil.which("hipcc") or os.path.join(rocm, "bin", "hipcc")
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; a ROCm toolchain is required to build")
    return path


def build_command(out_path: str = LIB_PATH) -> list:
    return ([hipcc()] + HIPCC_FLAGS + ["-I", INCLUDE, "-I", CSRC, "-o", out_path]
            + [os.path.join(CSRC, s) for s in SOURCES])


def build(verbose: bool = False) -> str:
    """Compile every source into ``libqm_attn.so`` (atomically replaced)."""
    tmp = LIB_PATH + f".tmp{os.getpid()}"
    cmd = build_command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    if verbose and res.stderr.strip():
        print(res.stderr, file=sys.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
