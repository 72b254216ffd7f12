"""Whole-output comparison of a GPU result with the fp64 oracle, in parallel.

TEST INFRASTRUCTURE.  For workloads too large for one CPU core (up to
B = 1, H = 32, N = 32768), every (batch, query head) is evaluated by the
oracle (``oracle.attention_fp64``, the plain definition) in a pool of worker
processes, each with single-threaded BLAS, one process per CPU this process
may keep busy.  A worker compares its head's exact outputs with the GPU's,
element by element, under the parity gate of ``tests/gpu_util.py`` (FP8
inputs: the rounding bound of ``tests/fp8_gate.py``) and returns statistics
only.  The inputs and the GPU outputs reach the workers through fork (shared
pages), so nothing of full size is copied.
"""
from __future__ import annotations

import multiprocessing as mp
import time

import numpy as np

from oracle import attention_fp64
from tests import fp8_gate
from tests.gpu_util import assert_stats, compare, say

# the job of the current pool (read by forked workers)
_JOB: dict = {}


def workers() -> int:
    """CPUs this process may keep busy (scheduler affinity capped by the cgroup
    CPU quota)."""
    import bench
    return bench.usable_cpus()[1]


def _decode_bits(bits: np.ndarray, dtype: str) -> np.ndarray:
    """16-bit output bit patterns -> fp64 (exact)."""
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _head(bh):
    from threadpoolctl import threadpool_limits
    j = _JOB
    b, h = bh
    q, k, v = j["q"], j["k"], j["v"]
    hk = h // (q.shape[1] // k.shape[1])
    with threadpool_limits(limits=1):
        Or, lr = attention_fp64(q[b:b + 1, h:h + 1], k[b:b + 1, hk:hk + 1], v[b:b + 1, hk:hk + 1],
                                j["scale"], j["causal"], j["dtype"], descale=j["descale"])
        Or, lr = Or[0, 0], lr[0, 0]
        Og = _decode_bits(j["o_bits"][b, h], j["out_dtype"])
        lg = j["lse"][b, h].astype(np.float64)
        bound = None
        if j["dtype"] == "e4m3":
            N = q.shape[2]
            bound = np.empty_like(Or)
            for r0 in range(0, N, 256):
                r1 = min(N, r0 + 256)
                bound[r0:r1] = fp8_gate.rounding_bound(q[b, h, r0:r1], k[b, hk], v[b, hk],
                                                       j["descale"], j["scale"], j["causal"],
                                                       np.arange(r0, r1), Or[r0:r1])
        st = compare(Og, lg, Or, lr, j["out_dtype"], bound=bound)
    st["head"] = (b, h)
    return st


def _merge(parts):
    out = {"n": 0, "nonfinite_o": 0, "nonfinite_lse": 0, "max_err": 0.0, "bad": 0,
           "over_tol": 0, "max_lse_err": 0.0}
    worst_excess = None
    for st in parts:
        for key in ("n", "nonfinite_o", "nonfinite_lse", "bad", "over_tol"):
            out[key] += st[key]
        out["max_err"] = max(out["max_err"], st["max_err"])
        if "worst" in st:
            idx, og, orf, e, bnd = st["worst"]
            if worst_excess is None or e - bnd > worst_excess:
                worst_excess = e - bnd
                out["worst"] = (st["head"] + idx, og, orf, e, bnd)
        if st["max_lse_err"] >= out["max_lse_err"]:
            out["max_lse_err"] = st["max_lse_err"]
            if "worst_lse" in st:
                idx, lg, lr = st["worst_lse"]
                out["worst_lse"] = (st["head"] + idx, lg, lr)
    return out


def full_compare(q, k, v, o_bits, lse, scale, causal, dtype, what, descale=None):
    """Compare every output of a GPU run with the oracle and assert the gate.

    ``q`` [B, H, N, d], ``k`` [B, Hkv, N, d], ``v`` [B, Hkv, N, dv]: the inputs
    as the oracle takes them (``dtype`` "f16", "bf16" or "e4m3" with
    ``descale`` = (q_scale, k_scale, v_scale)); ``o_bits`` [B, H, N, dv]
    uint16: the GPU's output bit patterns (bf16 for FP8 inputs); ``lse``
    [B, H, N] float32: the GPU's lse.  Returns the merged statistics.
    """
    B, H = q.shape[:2]
    out_dtype = "bf16" if dtype == "e4m3" else dtype
    heads = [(b, h) for b in range(B) for h in range(H)]
    n = max(1, min(workers(), len(heads)))
    _JOB.clear()
    _JOB.update(q=q, k=k, v=v, o_bits=o_bits, lse=lse, scale=scale, causal=causal, dtype=dtype,
                out_dtype=out_dtype, descale=descale)
    say(f"{what}: oracle over all {len(heads)} (batch, head) slices on {n} processes")
    t0 = last = time.perf_counter()
    parts = []
    try:
        with mp.get_context("fork").Pool(n) as pool:
            for st in pool.imap_unordered(_head, heads, chunksize=1):
                parts.append(st)
                now = time.perf_counter()
                if now - last > 10:
                    say(f"{what}: {len(parts)}/{len(heads)} slices compared "
                        f"({now - t0:.0f} s)")
                    last = now
    finally:
        _JOB.clear()
    st = _merge(parts)
    assert_stats(st, out_dtype, f"{what} (every element, {time.perf_counter() - t0:.1f} s)")
    return st


def gpu_bits(o) -> np.ndarray:
    """A 16-bit torch tensor's bit patterns on the host, as uint16."""
    import torch
    return o.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
