"""Build the plain-C client of the attention library (``tests/c_client.c``)
into ``tests/libqm_c_client.so``, linked against ``libqm_attn.so`` and the HIP
runtime.  Host code only: gcc with the HIP runtime headers, no device code.
Called by ``__graft_entry__.build()`` after the library itself."""
from __future__ import annotations

import os
import subprocess

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
SOURCE = os.path.join(TESTS, "c_client.c")
OUT = os.path.join(TESTS, "libqm_c_client.so")
PKG = os.path.join(ROOT, "paper_2506_12355_amd")


def build(verbose: bool = False) -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    tmp = OUT + f".tmp{os.getpid()}"
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-fPIC", "-shared",
           # the HIP runtime headers need the platform named when the compiler is not hipcc
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(rocm, "include"),
           "-I", os.path.join(ROOT, "include"), "-o", tmp, SOURCE,
           "-L", PKG, "-lqm_attn", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           # found relative to this file wherever the tree is copied
           "-Wl,-rpath,$ORIGIN/../paper_2506_12355_amd:" + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError(f"gcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
