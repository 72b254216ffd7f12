"""Helpers for the GPU parity tests: device transfer, the parity gate, reporting.

The gate (per element): |O_gpu - O_ref| <= tol + half an ulp of the storage
type at the output's magnitude, where tol is 2e-3 for fp16 and 1e-2 for bf16;
|lse_gpu - lse_ref| <= 1e-3.  The half ulp is the rounding of the exact value
to the 16-bit output type, which no storing kernel can avoid (a bf16 ulp is
already 3.1e-2 at |O| in [4, 8)).
"""
from __future__ import annotations

import numpy as np

TOL = {"f16": 2e-3, "bf16": 1e-2}
LSE_TOL = 1e-3
_MANT = {"f16": 10, "bf16": 7}
_EMIN = {"f16": -14, "bf16": -126}


def to_device(x: np.ndarray, dtype: str):
    import torch
    if dtype == "f16":
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda().view(torch.bfloat16)


def to_host64(t) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def half_ulp(x: np.ndarray, dtype: str) -> np.ndarray:
    a = np.abs(np.asarray(x, dtype=np.float64))
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.maximum(np.where(a > 0, e, _EMIN[dtype]), _EMIN[dtype])
    return np.ldexp(0.5, (e - _MANT[dtype]).astype(np.int64))


def check_close(O_gpu, lse_gpu, O_ref, lse_ref, dtype: str, what: str = ""):
    """Assert the parity gate; return (raw max-abs O error, max lse error)."""
    O_gpu = np.asarray(O_gpu, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    assert O_gpu.shape == O_ref.shape, (O_gpu.shape, O_ref.shape)
    assert np.all(np.isfinite(O_gpu)), f"{what}: non-finite O"
    assert np.all(np.isfinite(lse_gpu)), f"{what}: non-finite lse"
    err = np.abs(O_gpu - O_ref)
    bound = TOL[dtype] + np.maximum(half_ulp(O_ref, dtype), half_ulp(O_gpu, dtype))
    bad = err > bound
    if np.any(bad):
        idx = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(
            f"{what}: {int(bad.sum())} O elements outside the gate; worst at {idx}: "
            f"gpu={O_gpu[idx]!r} ref={O_ref[idx]!r} err={err[idx]:.3e} bound={bound[idx]:.3e}")
    lerr = np.abs(lse_gpu - lse_ref)
    if lerr.size and lerr.max() > LSE_TOL:
        idx = np.unravel_index(np.argmax(lerr), lerr.shape)
        raise AssertionError(f"{what}: lse err {lerr[idx]:.3e} at {idx}: "
                             f"gpu={lse_gpu[idx]!r} ref={lse_ref[idx]!r}")
    return float(err.max()) if err.size else 0.0, float(lerr.max()) if lerr.size else 0.0
