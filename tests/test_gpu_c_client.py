"""The C ABI driven from plain C (``tests/c_client.c``): hipMalloc'd buffers,
a stream created in C, hipMemcpy both ways, no torch on the call path.

Every entry point declared in include/qm_attn.h runs once through the client.
Its outputs must match the oracle under the usual gate and be byte-identical
to the Python binding's on the same inputs; an invalid argument must come back
as the documented status with the library's message.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64
from tests.gpu_util import check_close, half_ulp, to_device

pytestmark = pytest.mark.gpu

TESTS = os.path.dirname(os.path.abspath(__file__))
CLIENT = os.path.join(TESTS, "libqm_c_client.so")
ENTRY = {"fwd": 0, "gqa": 1, "mla": 2, "fp8": 3, "layout": 4, "fp8_layout": 5}
LN2 = math.log(2.0)


def load_client():
    if not os.path.exists(CLIENT):
        raise RuntimeError(f"{CLIENT} is missing: run __graft_entry__.build() first")
    lib = ctypes.CDLL(CLIENT)
    P, S, I, F = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_float
    lib.qmc_run.argtypes = [I, P, S, P, S, P, S, P, S, P, S, I, I, I, I, I, I, F, I, I, I,
                            F, F, F, ctypes.c_char_p, I]
    lib.qmc_run.restype = I
    return lib


@pytest.fixture(scope="module")
def client():
    import torch
    import paper_2506_12355_amd as qa
    assert torch.cuda.is_available()
    qa.load_library()
    return load_client(), qa


def run_c(lib, entry, q, k, v, o_elems, B, H, Hkv, N, d_qk, d_v, scale, causal, dtype=0,
          layout=0, scales=(1.0, 1.0, 1.0)):
    """One call through the C client; returns (status, message, o bits, lse)."""
    q, k, v = (np.ascontiguousarray(x) for x in (q, k, v))
    o = np.empty(o_elems, dtype=np.uint16)
    lse = np.empty(B * H * N, dtype=np.float32)
    msg = ctypes.create_string_buffer(256)
    st = lib.qmc_run(ENTRY[entry], q.ctypes.data, q.nbytes, k.ctypes.data, k.nbytes,
                     v.ctypes.data, v.nbytes, o.ctypes.data, o.nbytes, lse.ctypes.data,
                     lse.nbytes, B, H, Hkv, N, d_qk, d_v, scale, int(causal), dtype, layout,
                     *scales, msg, len(msg))
    return st, msg.value.decode(), o, lse


def bits_to_f64(bits, dtype):
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def same_bytes(o_c, lse_c, o_t, lse_t):
    import torch
    torch.cuda.synchronize()
    assert np.array_equal(o_c, o_t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                          .reshape(-1))
    assert np.array_equal(lse_c.view(np.uint32),
                          lse_t.view(torch.int32).cpu().numpy().view(np.uint32).reshape(-1))


@pytest.mark.parametrize("entry,dtype,B,H,Hkv,N,d,dv", [
    ("fwd", "f16", 2, 3, 3, 333, 64, 64),
    ("gqa", "bf16", 2, 6, 2, 200, 128, 128),
    ("mla", "f16", 1, 2, 2, 150, 192, 128),
])
def test_16bit_entries_from_c(client, entry, dtype, B, H, Hkv, N, d, dv):
    lib, qa = client
    q, k, v = si.make_qkv(B, H, N, d, dtype, seed=90 + N, Hkv=Hkv, dv=dv)
    scale = si.default_scale(d)
    code = qa.QM_F16 if dtype == "f16" else qa.QM_BF16
    for causal in (False, True):
        st, msg, o, lse = run_c(lib, entry, q, k, v, B * H * N * dv, B, H, Hkv, N, d, dv,
                                scale, causal, dtype=code)
        assert st == qa.QM_OK, msg
        O = bits_to_f64(o, dtype).reshape(B, H, N, dv)
        Or, lr = attention_fp64(q, k, v, scale, causal, dtype)
        check_close(O, lse.reshape(B, H, N), Or, lr, dtype, f"C {entry} causal={causal}")
        ot, lt = qa.fwd(*(to_device(x, dtype) for x in (q, k, v)), causal=causal, scale=scale)
        same_bytes(o, lse, ot, lt)


def test_layout_entry_from_c(client):
    lib, qa = client
    B, H, Hkv, N, d = 2, 4, 2, 257, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=95, Hkv=Hkv)
    tr = [np.swapaxes(x, 1, 2) for x in (q, k, v)]     # [B][N][heads][d]
    scale = si.default_scale(d)
    for causal in (False, True):
        st, msg, o, lse = run_c(lib, "layout", *tr, B * N * H * d, B, H, Hkv, N, d, d, scale,
                                causal, dtype=qa.QM_BF16, layout=qa.QM_BNHD)
        assert st == qa.QM_OK, msg
        O = np.swapaxes(bits_to_f64(o, "bf16").reshape(B, N, H, d), 1, 2)
        Or, lr = attention_fp64(q, k, v, scale, causal, "bf16")
        check_close(O, lse.reshape(B, H, N), Or, lr, "bf16", f"C layout causal={causal}")
        ot, lt = qa.fwd(*(to_device(x, "bf16") for x in tr), causal=causal, scale=scale,
                        layout="bnhd")
        same_bytes(o, lse, ot, lt)


@pytest.mark.parametrize("entry,H,Hkv,N,layout", [
    ("fp8", 3, 3, 333, "bhnd"),
    ("fp8_layout", 4, 2, 129, "bnhd"),
])
def test_fp8_entries_from_c(client, entry, H, Hkv, N, layout):
    """Exact-weight FP8 inputs: the oracle's value up to fp32 summation and
    the bf16 output rounding."""
    import torch
    lib, qa = client
    B, d = 2, 128
    q8, k8, v8 = si.make_qkv_fp8_dyadic(B, H, N, d, seed=96 + N, v_binade=True, Hkv=Hkv)
    scales = (0.5, 2.0, 0.0123)
    bnhd = layout == "bnhd"
    lay = (lambda x: np.swapaxes(x, 1, 2)) if bnhd else (lambda x: x)
    for causal in (False, True):
        st, msg, o, lse = run_c(lib, entry, *(lay(x) for x in (q8, k8, v8)), B * H * N * d, B,
                                H, Hkv, N, d, d, LN2, causal,
                                layout=qa.QM_BNHD if bnhd else qa.QM_BHND, scales=scales)
        assert st == qa.QM_OK, msg
        O = bits_to_f64(o, "bf16").reshape((B, N, H, d) if bnhd else (B, H, N, d))
        O = np.swapaxes(O, 1, 2) if bnhd else O
        Or, lr = attention_fp64(q8, k8, v8, LN2, causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        bound = (half_ulp(Or, "bf16")
                 + (2 * (N + 128) * 2.0 ** -24 + 1e-5) * PV)
        assert np.all(np.abs(O - Or) <= bound), float(np.max(np.abs(O - Or) - bound))
        assert np.max(np.abs(lse.reshape(B, H, N) - lr)) <= 1e-3
        codes = [torch.from_numpy(np.ascontiguousarray(lay(x))).cuda().view(torch.float8_e4m3fn)
                 for x in (q8, k8, v8)]
        ot, lt = qa.fwd_fp8(*codes, scales, causal=causal, scale=LN2, layout=layout)
        same_bytes(o, lse, ot, lt)


def test_invalid_argument_from_c(client):
    """A bad head dimension comes back as QM_ERR_HEADDIM with the library's
    text, after the client's buffers were allocated on the device."""
    lib, qa = client
    q, k, v = si.make_qkv(1, 2, 64, 96, "f16", seed=97)
    st, msg, o, lse = run_c(lib, "fwd", q, k, v, 2 * 64 * 96, 1, 2, 2, 64, 96, 96, 0.1, False)
    assert st == qa.QM_ERR_HEADDIM
    assert msg == qa.strerror(qa.QM_ERR_HEADDIM)
