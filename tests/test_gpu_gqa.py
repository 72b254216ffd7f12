"""GPU parity for grouped-query and multi-query attention (``qm_attn_fwd_gqa``).

H query heads share Hkv key/value heads; query head h reads key/value head
h // (H / Hkv).  The oracle maps heads the same way and is otherwise the
multi-head definition.  Small workloads are compared in full, the long ones
(the appendix table's LLM head configurations and multi-query attention at
N = 8192) on sampled rows and then on every element, with the oracle spread
over processes.  Independently of the oracle, a grouped call must
equal, byte for byte, the multi-head call on K and V with every head repeated.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64, attention_rows_fp64
from tests import oracle_pool
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


@pytest.mark.parametrize("name", ["gqa_b2_h8_kv2_n1000_d64_f16", "mqa_b2_h6_kv1_n777_d128_bf16"])
def test_small_gqa_workloads_full(qa, name):
    import torch
    w = si.WORKLOADS[name]
    q, k, v = w.inputs()
    assert k.shape[1] == w.kv_heads < w.H
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    for causal in w.causal:
        _say(f"case {name} causal={causal}")
        o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale)
        torch.cuda.synchronize()
        Or, lr = attention_fp64(q, k, v, w.scale, causal, w.dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, w.dtype, f"{name} causal={causal}")


def _sample_rows(w, n, seed):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 63, 64, 255, 256, w.N // 2, w.N - 257, w.N - 2, w.N - 1]
    rows = []
    for t in range(n):
        b = int(rng.integers(w.B))
        h = int(rng.integers(w.H))
        i = fixed[t] if t < len(fixed) else int(rng.integers(w.N))
        rows.append((b, h, i))
    return rows


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,causal", [
    ("gqa_b2_h64_kv8_n8192_d128_bf16_causal", True),
    ("gqa_b2_h128_kv8_n8192_d128_bf16_causal", True),
    ("mqa_b2_h32_kv1_n8192_d128_bf16", False),
    ("mqa_b2_h32_kv1_n8192_d128_bf16", True),
])
def test_long_gqa_workloads_sampled(qa, name, causal):
    import torch
    w = si.WORKLOADS[name]
    _say(f"case {name} causal={causal}: drawing inputs")
    q, k, v = w.inputs()
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    _say(f"case {name} causal={causal}: running")
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    vmax = float(tv.abs().amax(dim=2).float().max())
    assert float(o.abs().float().max()) <= vmax * (1 + 2 ** -7)
    rows = _sample_rows(w, 128, seed=3)
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    _say(f"case {name} causal={causal}: oracle on {len(rows)} rows")
    Or, lr = attention_rows_fp64(q, k, v, w.scale, causal, w.dtype, rows)
    check_close(to_host64(o[ix]), to_host64(lse[ix]), Or, lr, w.dtype,
                f"{name} causal={causal} sampled rows")
    # then every output element, the oracle spread over processes
    bits, L = oracle_pool.gpu_bits(o), lse.cpu().numpy()
    del o, lse, tq, tk, tv
    oracle_pool.full_compare(q, k, v, bits, L, w.scale, causal, w.dtype,
                             f"{name} causal={causal}")


@pytest.mark.parametrize("N", [1, 65, 333, 1000])
@pytest.mark.parametrize("H,Hkv", [(4, 1), (4, 2), (6, 3), (16, 2)])
@pytest.mark.parametrize("dtype,d", [("f16", 64), ("bf16", 128)])
def test_gqa_equals_mha_on_repeated_heads(qa, H, Hkv, dtype, d, N):
    import torch
    q, k, v = si.make_qkv(2, H, N, d, dtype, seed=H * 31 + Hkv * 7 + N, Hkv=Hkv)
    tq, tk, tv = (to_device(x, dtype) for x in (q, k, v))
    tkr = tk.repeat_interleave(H // Hkv, dim=1).contiguous()
    tvr = tv.repeat_interleave(H // Hkv, dim=1).contiguous()
    for causal in (False, True):
        _say(f"case repeated heads H={H} Hkv={Hkv} N={N} d={d} {dtype} causal={causal}")
        o, lse = qa.fwd(tq, tk, tv, causal=causal)
        o2, l2 = qa.fwd(tq, tkr, tvr, causal=causal)
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o2.view(torch.int16))
        assert torch.equal(lse.view(torch.int32), l2.view(torch.int32))
    if N == 333:
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), True, dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, dtype, f"GQA H={H} Hkv={Hkv} causal")


def test_gqa_entry_with_all_heads_is_mha(qa):
    """qm_attn_fwd_gqa with Hkv = H runs the same computation as qm_attn_fwd."""
    import torch
    B, H, N, d = 2, 3, 200, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=77)
    tq, tk, tv = (to_device(x, "bf16") for x in (q, k, v))
    stream = torch.cuda.current_stream().cuda_stream
    for causal in (0, 1):
        outs = []
        for gqa in (False, True):
            o = torch.empty_like(tq)
            lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
            args = (tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), o.data_ptr(), lse.data_ptr())
            scale = si.default_scale(d)
            if gqa:
                st = qa.qm_attn_fwd_gqa(*args, B, H, H, N, d, scale, causal, stream, qa.QM_BF16)
            else:
                st = qa.qm_attn_fwd(*args, B, H, N, d, scale, causal, stream, qa.QM_BF16)
            assert st == qa.QM_OK
            outs.append((o, lse))
        torch.cuda.synchronize()
        assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
        assert torch.equal(outs[0][1].view(torch.int32), outs[1][1].view(torch.int32))


def test_gqa_inputs_read_only_within_bounds(qa):
    """NaN right after the last key/value head (Hkv of them) and the last query
    head never reaches the outputs."""
    import torch
    B, H, Hkv, N, d = 2, 4, 2, 197, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=43, Hkv=Hkv)
    views = []
    for x in (q, k, v):
        t = to_device(x, "bf16").reshape(-1)
        buf = torch.full((t.numel() + 2 * 64 * d,), float("nan"), dtype=t.dtype, device="cuda")
        buf[:t.numel()] = t
        views.append(buf[:t.numel()].view(x.shape))
    for causal in (False, True):
        o, lse = qa.fwd(*views, causal=causal)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), causal, "bf16")
        check_close(to_host64(o), to_host64(lse), Or, lr, "bf16", f"guarded GQA causal={causal}")
