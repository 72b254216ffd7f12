"""GPU parity for the [B][N][heads][d] layout (``qm_attn_fwd_layout`` with
QM_BNHD): the same operation as the [B][H][N][d] entry points on tensors whose
heads sit side by side per token.

Inputs are drawn in [B][H][N][d] (the oracle's layout) and transposed for the
device, and outputs are transposed back.  The results must match the oracle
under the usual gate, and be byte-identical to the [B][H][N][d] entry
points' on the same values (the kernels do the same arithmetic in the same
order; only addresses differ).
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64, attention_rows_fp64
from tests.gpu_util import check_close, to_device, to_host64

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def qa():
    import torch
    import paper_2506_12355_amd as qa
    assert torch.cuda.is_available()
    qa.load_library()
    return qa


def _bnhd(x):
    """[B][H][N][d] numpy array -> contiguous [B][N][H][d]."""
    return np.ascontiguousarray(np.swapaxes(x, 1, 2))


def _case(qa, q, k, v, dtype, causal, what):
    import torch
    scale = si.default_scale(q.shape[-1])
    tq, tk, tv = (to_device(_bnhd(x), dtype) for x in (q, k, v))
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=scale, layout="bnhd")
    torch.cuda.synchronize()
    assert tuple(o.shape) == (q.shape[0], q.shape[2], q.shape[1], v.shape[-1])
    O = np.swapaxes(to_host64(o), 1, 2)
    Or, lr = attention_fp64(q, k, v, scale, causal, dtype)
    check_close(O, to_host64(lse), Or, lr, dtype, what)
    # the same values through the [B][H][N][d] entry points: byte for byte
    ob, lb = qa.fwd(*(to_device(x, dtype) for x in (q, k, v)), causal=causal, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(o.transpose(1, 2).contiguous().view(torch.int16), ob.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lb.view(torch.int32))


@pytest.mark.parametrize("N", [1, 65, 333, 1000])
@pytest.mark.parametrize("dtype,d", [("f16", 64), ("bf16", 128)])
def test_bnhd_multi_head(qa, N, dtype, d):
    q, k, v = si.make_qkv(2, 3, N, d, dtype, seed=60 + N)
    for causal in (False, True):
        _say(f"case BNHD MHA N={N} {dtype} d={d} causal={causal}")
        _case(qa, q, k, v, dtype, causal, f"BNHD N={N} d={d} causal={causal}")


@pytest.mark.parametrize("H,Hkv", [(4, 2), (6, 1)])
def test_bnhd_grouped_query(qa, H, Hkv):
    q, k, v = si.make_qkv(2, H, 777, 128, "bf16", seed=61, Hkv=Hkv)
    for causal in (False, True):
        _say(f"case BNHD GQA H={H} Hkv={Hkv} causal={causal}")
        _case(qa, q, k, v, "bf16", causal, f"BNHD GQA {H}/{Hkv} causal={causal}")


def test_bnhd_bounds_and_outputs(qa):
    """NaN right after each input tensor never reaches the outputs (rows past
    the end of the sequence read as zeros even though a head's rows are H
    rows apart); NaN-poisoned outputs are fully overwritten and the guard
    zones around o stay untouched."""
    import torch
    B, H, N, d = 2, 3, 197, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=62)
    views = []
    for x in (q, k, v):
        t = to_device(_bnhd(x), "bf16").reshape(-1)
        buf = torch.full((t.numel() + 2 * 64 * H * d,), float("nan"), dtype=t.dtype,
                         device="cuda")
        buf[:t.numel()] = t
        views.append(buf[:t.numel()].view(B, N, H, d))
    G = 256
    for causal in (False, True):
        _say(f"case BNHD guarded causal={causal}")
        obuf = torch.full((B * N * H * d + 2 * G,), float("nan"), dtype=torch.bfloat16,
                          device="cuda")
        obuf[:G] = 7.0
        obuf[-G:] = 7.0
        o = obuf[G:G + B * N * H * d].view(B, N, H, d)
        o, lse = qa.fwd(*views, causal=causal, out=o, layout="bnhd")
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        assert bool((obuf[:G] == 7.0).all()) and bool((obuf[-G:] == 7.0).all())
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), causal, "bf16")
        check_close(np.swapaxes(to_host64(o), 1, 2), to_host64(lse), Or, lr, "bf16",
                    f"BNHD guarded causal={causal}")


@pytest.mark.parametrize("causal", [False, True])
def test_bnhd_bench_shape_sampled(qa, causal):
    """B = 2, H = 32, N = 8192, d = 128 in the [B][N][H][d] layout, on sampled
    rows, and byte-identical to the [B][H][N][d] launch."""
    import torch
    w = si.WORKLOADS["mha_b2_h32_n8192_d128_bf16"]
    q, k, v = w.inputs()
    tq, tk, tv = (to_device(_bnhd(x), "bf16") for x in (q, k, v))
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale, layout="bnhd")
    ob, lb = qa.fwd(*(to_device(x, "bf16") for x in (q, k, v)), causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    assert torch.equal(o.transpose(1, 2).contiguous().view(torch.int16), ob.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lb.view(torch.int32))
    rng = np.random.default_rng(63)
    rows = [(int(rng.integers(2)), int(rng.integers(32)), int(rng.integers(8192)))
            for _ in range(48)] + [(0, 0, 0), (1, 31, 8191)]
    O = np.array([to_host64(o[b, i, h]) for b, h, i in rows])
    L = np.array([float(lse[b, h, i]) for b, h, i in rows])
    Or, lr = attention_rows_fp64(q, k, v, w.scale, causal, "bf16", rows)
    check_close(O, L, Or, lr, "bf16", f"BNHD bench shape causal={causal}")
