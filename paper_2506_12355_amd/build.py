"""Build the gfx950 attention library in place: ``libqm_attn.so`` beside this file.

Usage: ``python -m paper_2506_12355_amd.build`` (or call :func:`build`).  It
always recompiles.  hipcc cross-compiles for gfx950 without a GPU present.

It also builds ``libqm_attn_debug.so``, the same sources with
``-DQM_DEBUG_SYNC``: a barrier after every key block on top of the K/V ring
protocol's own.  The tests check that it gives the same bytes as the release
library; nothing else loads it.
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
DEBUG_LIB_PATH = os.path.join(PKG_DIR, "libqm_attn_debug.so")

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


def build_command(out_path: str = LIB_PATH, debug_sync: bool = False) -> list:
    return ([hipcc()] + HIPCC_FLAGS + (["-DQM_DEBUG_SYNC"] if debug_sync else [])
            + ["-I", INCLUDE, "-I", CSRC, "-o", out_path]
            + [os.path.join(CSRC, s) for s in SOURCES])


def build(verbose: bool = False) -> str:
    """Compile every source into ``libqm_attn.so`` and ``libqm_attn_debug.so``
    (two hipcc processes at once; each library atomically replaced)."""
    jobs = []
    for path, debug in ((LIB_PATH, False), (DEBUG_LIB_PATH, True)):
        tmp = path + f".tmp{os.getpid()}"
        cmd = build_command(tmp, debug_sync=debug)
        if verbose:
            print(" ".join(cmd), flush=True)
        jobs.append((path, tmp, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                 stderr=subprocess.PIPE, text=True)))
    failed = []
    for path, tmp, proc in jobs:
        out, err = proc.communicate()
        if proc.returncode != 0:
            if os.path.exists(tmp):
                os.remove(tmp)
            failed.append(f"hipcc failed for {path} ({proc.returncode}):\n{out}\n{err}")
            continue
        if verbose and err.strip():
            print(err, file=sys.stderr)
        os.replace(tmp, path)
    if failed:
        raise RuntimeError("\n".join(failed))
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
