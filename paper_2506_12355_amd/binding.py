"""ctypes binding of the C-ABI attention library (include/qm_attn.h).

Argument marshalling only: every step of the attention forward runs in the
gfx950 kernels.  PyTorch supplies device memory and the current HIP stream.
There is no fallback: if ``libqm_attn.so`` is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
import threading

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libqm_attn.so")
DEBUG_LIB_PATH = os.path.join(PKG_DIR, "libqm_attn_debug.so")

# qm_dtype_t
QM_F16 = 0
QM_BF16 = 1

# qm_layout_t
QM_BHND = 0
QM_BNHD = 1

# status codes
QM_OK = 0
QM_ERR_NULL = -1
QM_ERR_SHAPE = -2
QM_ERR_HEADDIM = -3
QM_ERR_DTYPE = -4
QM_ERR_SCALE = -5
QM_ERR_ALIAS = -6
QM_ERR_CAUSAL = -7
QM_ERR_LAUNCH = -8
QM_ERR_UNSUPPORTED = -9
QM_ERR_LAYOUT = -10
QM_ERR_TILE = -11

_lib = None
_lock = threading.Lock()


class QmAttnError(RuntimeError):
    """A non-zero status from the C library."""

    def __init__(self, status: int, message: str):
        super().__init__(f"qm_attn_fwd failed with status {status}: {message}")
        self.status = status


def _declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    """Argument and result types of every entry point of ``include/qm_attn.h``."""
    lib.qm_attn_fwd.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
    ]
    lib.qm_attn_fwd.restype = ctypes.c_int
    lib.qm_attn_fwd_gqa.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
    ]
    lib.qm_attn_fwd_gqa.restype = ctypes.c_int
    lib.qm_attn_fwd_mla.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
    ]
    lib.qm_attn_fwd_mla.restype = ctypes.c_int
    lib.qm_attn_fwd_fp8.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int,
        ctypes.c_void_p,
    ]
    lib.qm_attn_fwd_fp8.restype = ctypes.c_int
    lib.qm_attn_fwd_layout.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
    ]
    lib.qm_attn_fwd_layout.restype = ctypes.c_int
    lib.qm_attn_fwd_fp8_layout.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int,
        ctypes.c_void_p, ctypes.c_int,
    ]
    lib.qm_attn_fwd_fp8_layout.restype = ctypes.c_int
    lib.qm_attn_set_tile_rows.argtypes = [ctypes.c_int]
    lib.qm_attn_set_tile_rows.restype = ctypes.c_int
    lib.qm_attn_strerror.argtypes = [ctypes.c_int]
    lib.qm_attn_strerror.restype = ctypes.c_char_p
    return lib


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load (once) and return the HIP library; raise if it has not been built."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        _lib = open_library(path)
        return _lib


def open_library(path: str) -> ctypes.CDLL:
    """A separate handle on a build of the library at ``path`` (the tests use
    it for the checking build, ``libqm_attn_debug.so``); raises if missing."""
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: the HIP attention library has not been built "
            "(run `python -m paper_2506_12355_amd.build`)")
    return _declare(ctypes.CDLL(path))


def strerror(status: int) -> str:
    return load_library().qm_attn_strerror(int(status)).decode()


def set_tile_rows(rows: int) -> None:
    """Query rows per workgroup for later calls: 0 (chosen from the shape, the
    default), 128 or 256.  Outputs are byte-identical either way; only speed
    changes (``qm_attn_set_tile_rows``)."""
    status = load_library().qm_attn_set_tile_rows(int(rows))
    if status != QM_OK:
        raise QmAttnError(status, strerror(status))


def qm_attn_fwd(q, k, v, o, lse, B, H, N, d, scale, causal, stream, dtype) -> int:
    """The C entry point with plain integers for pointers; returns the status."""
    return load_library().qm_attn_fwd(q, k, v, o, lse, int(B), int(H), int(N), int(d),
                                      float(scale), int(causal), stream, int(dtype))


def qm_attn_fwd_layout(q, k, v, o, lse, B, H, Hkv, N, d_qk, d_v, scale, causal, stream, dtype,
                       layout) -> int:
    """The general 16-bit C entry point (layout argument) with plain integers
    for pointers; returns the status."""
    return load_library().qm_attn_fwd_layout(q, k, v, o, lse, int(B), int(H), int(Hkv), int(N),
                                             int(d_qk), int(d_v), float(scale), int(causal),
                                             stream, int(dtype), int(layout))


def qm_attn_fwd_gqa(q, k, v, o, lse, B, H, Hkv, N, d, scale, causal, stream, dtype) -> int:
    """The grouped-query C entry point with plain integers for pointers; returns the status."""
    return load_library().qm_attn_fwd_gqa(q, k, v, o, lse, int(B), int(H), int(Hkv), int(N),
                                          int(d), float(scale), int(causal), stream, int(dtype))


def qm_attn_fwd_mla(q, k, v, o, lse, B, H, N, d_qk, d_v, scale, causal, stream, dtype) -> int:
    """The unequal-head-dimension C entry point with plain integers for pointers."""
    return load_library().qm_attn_fwd_mla(q, k, v, o, lse, int(B), int(H), int(N), int(d_qk),
                                          int(d_v), float(scale), int(causal), stream, int(dtype))


def qm_attn_fwd_fp8(q, k, v, o, lse, B, H, N, d, q_scale, k_scale, v_scale, scale, causal,
                    stream) -> int:
    """The FP8 C entry point with plain integers for pointers; returns the status."""
    return load_library().qm_attn_fwd_fp8(q, k, v, o, lse, int(B), int(H), int(N), int(d),
                                          float(q_scale), float(k_scale), float(v_scale),
                                          float(scale), int(causal), stream)


def fwd_fp8(q, k, v, scales, causal: bool = False, scale: float | None = None, out=None,
            lse=None, stream=None, layout: str = "bhnd"):
    """FP8 attention forward: q is [B, H, N, d], k and v [B, Hkv, N, d] (Hkv
    dividing H: grouped-query attention when Hkv < H) tensors of OCP E4M3 codes
    (``torch.float8_e4m3fn`` or ``uint8``) on a ROCm device; ``scales`` holds
    the three per-tensor factors (q_scale, k_scale, v_scale).  With
    ``layout="bnhd"`` the tensors are [B, N, heads, d] instead.  Returns
    (o, lse): o bf16 shaped like q, lse float32 [B, H, N] in either layout.
    ``scale`` defaults to 1/sqrt(d) rounded to float32.  Multi-head
    [B, H, N, d] calls go to ``qm_attn_fwd_fp8``, the others to
    ``qm_attn_fwd_fp8_layout``."""
    import torch

    if layout not in ("bhnd", "bnhd"):
        raise ValueError(f"layout must be 'bhnd' or 'bnhd', not {layout!r}")
    bnhd = layout == "bnhd"
    names = "[B, N, H, d]" if bnhd else "[B, H, N, d]"

    def shape(t):   # (B, heads, N, d) whatever the layout
        s = tuple(t.shape)
        return (s[0], s[2], s[1], s[3]) if bnhd else s

    for t in (q, k, v):
        if t.dim() != 4:
            raise ValueError(f"q, k and v must have shape {names}")
        if t.dtype not in (torch.uint8, torch.float8_e4m3fn):
            raise TypeError("FP8 inputs must be float8_e4m3fn or uint8 codes")
        if not t.is_cuda or t.device != q.device or not t.is_contiguous():
            raise ValueError("q, k and v must be contiguous tensors on one ROCm device")
    if shape(v) != shape(k) or shape(k)[0] != shape(q)[0] or shape(k)[2:] != shape(q)[2:]:
        raise ValueError("k and v must hold Hkv heads matching q in B, N and d")
    B, H, N, d = shape(q)
    Hkv = shape(k)[1]
    if scale is None:
        scale = float(torch.tensor(1.0 / d ** 0.5, dtype=torch.float32))
    if out is None:
        out = torch.empty(tuple(q.shape), dtype=torch.bfloat16, device=q.device)
    elif out.shape != q.shape or out.dtype != torch.bfloat16 or not out.is_contiguous():
        raise ValueError("out must be a contiguous bfloat16 tensor shaped like q")
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    elif lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 tensor of shape [B, H, N]")
    _check_outputs_on(q.device, out, lse)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    qs, ks, vs = (float(t) for t in scales)
    with torch.cuda.device(q.device):
        if bnhd or Hkv != H:
            status = qm_attn_fwd_fp8_layout(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                            out.data_ptr(), lse.data_ptr(), B, H, Hkv, N, d,
                                            qs, ks, vs, scale, 1 if causal else 0,
                                            stream.cuda_stream, QM_BNHD if bnhd else QM_BHND)
        else:
            status = qm_attn_fwd_fp8(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                     lse.data_ptr(), B, H, N, d, qs, ks, vs, scale,
                                     1 if causal else 0, stream.cuda_stream)
    if status != QM_OK:
        raise QmAttnError(status, strerror(status))
    return out, lse


def qm_attn_fwd_fp8_layout(q, k, v, o, lse, B, H, Hkv, N, d, q_scale, k_scale, v_scale, scale,
                           causal, stream, layout) -> int:
    """The general FP8 C entry point (key/value heads and layout as arguments)
    with plain integers for pointers; returns the status."""
    return load_library().qm_attn_fwd_fp8_layout(
        q, k, v, o, lse, int(B), int(H), int(Hkv), int(N), int(d), float(q_scale),
        float(k_scale), float(v_scale), float(scale), int(causal), stream, int(layout))


def _check_outputs_on(device, out, lse) -> None:
    """The kernel writes o and lse through device pointers: both must live on
    the inputs' device (a host tensor's address would be written by the GPU)."""
    for name, t in (("out", out), ("lse", lse)):
        if not t.is_cuda or t.device != device:
            raise ValueError(f"{name} must be on the inputs' device {device}, not {t.device}")


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float16:
        return QM_F16
    if t.dtype == torch.bfloat16:
        return QM_BF16
    raise TypeError(f"q, k, v must be float16 or bfloat16, not {t.dtype}")


def fwd(q, k, v, causal: bool = False, scale: float | None = None, out=None, lse=None,
        stream=None, layout: str = "bhnd"):
    """Attention forward on torch tensors on a ROCm device.

    q is [B, H, N, d]; k is [B, Hkv, N, d] and v [B, Hkv, N, dv] with Hkv
    dividing H.  Hkv = H and dv = d: multi-head attention (``qm_attn_fwd``);
    Hkv < H: grouped-query or multi-query attention (``qm_attn_fwd_gqa``);
    dv < d (d = 192, dv = 128, Hkv = H): the MLA shape (``qm_attn_fwd_mla``).
    With ``layout="bnhd"`` the tensors are [B, N, heads, width] instead (q
    [B, N, H, d], k [B, N, Hkv, d], v [B, N, Hkv, dv], o [B, N, H, dv];
    ``qm_attn_fwd_layout``).  Returns (o, lse): o of q's dtype, lse float32
    [B, H, N] in either layout.  ``scale`` defaults to 1/sqrt(d) rounded to
    float32.  ``stream`` defaults to the current stream of q's device.
    """
    import torch

    if layout not in ("bhnd", "bnhd"):
        raise ValueError(f"layout must be 'bhnd' or 'bnhd', not {layout!r}")
    bnhd = layout == "bnhd"
    names = "[B, N, H, d]" if bnhd else "[B, H, N, d]"
    if q.dim() != 4:
        raise ValueError(f"q must have shape {names}")

    def shape(t):   # (B, heads, N, width) whatever the layout
        s = tuple(t.shape)
        return (s[0], s[2], s[1], s[3]) if bnhd else s

    if k.dim() != 4 or v.dim() != 4 or shape(v)[:3] != shape(k)[:3]:
        raise ValueError("k must hold Hkv heads of width d and v Hkv heads of width dv")
    if shape(k)[0] != shape(q)[0] or shape(k)[2:] != shape(q)[2:]:
        raise ValueError("k must match q in B, N and d")
    if not (q.is_cuda and k.is_cuda and v.is_cuda):
        raise ValueError("q, k and v must be on a ROCm device")
    if not (q.device == k.device == v.device):
        raise ValueError("q, k and v must be on the same device")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k and v must have the same dtype")
    if not (q.is_contiguous() and k.is_contiguous() and v.is_contiguous()):
        raise ValueError(f"q, k and v must be contiguous {names}")
    B, H, N, d = shape(q)
    dv = shape(v)[3]
    Hkv = shape(k)[1]
    code = _dtype_code(q)
    if scale is None:
        scale = float(torch.tensor(1.0 / d ** 0.5, dtype=torch.float32))
    oshape = (B, N, H, dv) if bnhd else (B, H, N, dv)
    if out is None:
        out = torch.empty(oshape, dtype=q.dtype, device=q.device)
    elif tuple(out.shape) != oshape or out.dtype != q.dtype or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous {list(oshape)} tensor of q's dtype")
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    elif lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 tensor of shape [B, H, N]")
    _check_outputs_on(q.device, out, lse)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    with torch.cuda.device(q.device):
        if bnhd:
            status = qm_attn_fwd_layout(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                        out.data_ptr(), lse.data_ptr(), B, H, Hkv, N, d, dv,
                                        scale, 1 if causal else 0, stream.cuda_stream, code,
                                        QM_BNHD)
        elif dv != d:
            if Hkv != H:
                raise ValueError("unequal head dimensions need as many key/value heads as query heads")
            status = qm_attn_fwd_mla(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                     lse.data_ptr(), B, H, N, d, dv, scale, 1 if causal else 0,
                                     stream.cuda_stream, code)
        elif Hkv == H:
            status = qm_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                 lse.data_ptr(), B, H, N, d, scale, 1 if causal else 0,
                                 stream.cuda_stream, code)
        else:
            status = qm_attn_fwd_gqa(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                     lse.data_ptr(), B, H, Hkv, N, d, scale,
                                     1 if causal else 0, stream.cuda_stream, code)
    if status != QM_OK:
        raise QmAttnError(status, strerror(status))
    return out, lse
