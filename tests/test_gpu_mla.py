"""GPU parity for the MLA shape (``qm_attn_fwd_mla``): queries and keys 192
wide (head dimension 128 plus a 64-wide RoPE part), values and outputs 128.

The oracle computes the definition with the scores over all 192 columns.
Every workload is compared in full; the long ones (including the
DeepSeek-V3-sized one: 128 heads, N = 8192, causal) first on sampled rows,
then on every element with the oracle spread over processes.  Independently of the
oracle: with the last 64 query/key columns zero, the result must equal the
128-wide multi-head kernel's byte for byte (the extra k-steps add exact zeros).
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


def _run(qa, q, k, v, dtype, causal, scale):
    import torch
    tq, tk, tv = (to_device(x, dtype) for x in (q, k, v))
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=scale)
    torch.cuda.synchronize()
    return o, lse


@pytest.mark.parametrize("name", ["mla_b2_h4_n777_d192_dv128_f16"])
def test_small_mla_workload_full(qa, name):
    w = si.WORKLOADS[name]
    q, k, v = w.inputs()
    assert q.shape[-1] == 192 and v.shape[-1] == 128
    for causal in w.causal:
        _say(f"case {name} causal={causal}")
        o, lse = _run(qa, q, k, v, w.dtype, causal, w.scale)
        assert tuple(o.shape) == (w.B, w.H, w.N, 128)
        Or, lr = attention_fp64(q, k, v, w.scale, causal, w.dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, w.dtype, f"{name} causal={causal}")


@pytest.mark.parametrize("N", [1, 63, 65, 129, 255, 1000])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_mla_edge_lengths(qa, N, dtype):
    q, k, v = si.make_qkv(1, 3, N, 192, dtype, seed=N + 191, dv=128)
    for causal in (False, True):
        _say(f"case MLA edge N={N} {dtype} causal={causal}")
        o, lse = _run(qa, q, k, v, dtype, causal, si.default_scale(192))
        Or, lr = attention_fp64(q, k, v, si.default_scale(192), causal, dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, dtype, f"MLA N={N} causal={causal}")


def _sample_rows(w, n, seed):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 63, 64, 255, 256, w.N // 2, w.N - 257, w.N - 2, w.N - 1]
    return [(int(rng.integers(w.B)), int(rng.integers(w.H)),
             fixed[t] if t < len(fixed) else int(rng.integers(w.N))) for t in range(n)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,causal", [
    ("mla_b1_h16_n4096_d192_dv128_bf16", False),
    ("mla_b1_h16_n4096_d192_dv128_bf16", True),
    ("mla_b2_h128_n8192_d192_dv128_bf16_causal", True),
])
def test_long_mla_workloads_sampled(qa, name, causal):
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
    rows = _sample_rows(w, 128, seed=4)
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


@pytest.mark.parametrize("N", [200, 1000])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_zero_rope_part_equals_mha(qa, N, dtype):
    import torch
    q, k, v = si.make_qkv(2, 3, N, 192, dtype, seed=N + 3, dv=128)
    q[..., 128:] = 0
    k[..., 128:] = 0
    scale = si.default_scale(192)
    for causal in (False, True):
        _say(f"case zero RoPE part N={N} {dtype} causal={causal}")
        o, lse = _run(qa, q, k, v, dtype, causal, scale)
        o2, l2 = _run(qa, np.ascontiguousarray(q[..., :128]), np.ascontiguousarray(k[..., :128]),
                      v, dtype, causal, scale)
        assert torch.equal(o.view(torch.int16), o2.view(torch.int16))
        assert torch.equal(lse.view(torch.int32), l2.view(torch.int32))


def test_mla_inputs_read_only_within_bounds(qa):
    """NaN right after the last head of Q, K (192 wide) and V (128 wide) never
    reaches the outputs; NaN-poisoned outputs are fully overwritten and their
    guard zones untouched."""
    import torch
    B, H, N = 2, 2, 197
    q, k, v = si.make_qkv(B, H, N, 192, "bf16", seed=41, dv=128)
    views = []
    for x in (q, k, v):
        t = to_device(x, "bf16").reshape(-1)
        buf = torch.full((t.numel() + 2 * 64 * 192,), float("nan"), dtype=t.dtype, device="cuda")
        buf[:t.numel()] = t
        views.append(buf[:t.numel()].view(x.shape))
    G = 256
    for causal in (False, True):
        _say(f"case guarded MLA inputs causal={causal}")
        obuf = torch.full((B * H * N * 128 + 2 * G,), float("nan"), dtype=torch.bfloat16,
                          device="cuda")
        obuf[:G] = 7.0
        obuf[-G:] = 7.0
        o = obuf[G:G + B * H * N * 128].view(B, H, N, 128)
        o, lse = qa.fwd(*views, causal=causal, scale=si.default_scale(192), out=o)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        assert bool((obuf[:G] == 7.0).all()) and bool((obuf[-G:] == 7.0).all())
        Or, lr = attention_fp64(q, k, v, si.default_scale(192), causal, "bf16")
        check_close(to_host64(o), to_host64(lse), Or, lr, "bf16", f"guarded MLA causal={causal}")


def test_mla_bit_stable_across_runs(qa):
    import torch
    q, k, v = si.make_qkv(2, 3, 555, 192, "f16", seed=42, dv=128)
    tq, tk, tv = (to_device(x, "f16") for x in (q, k, v))
    for causal in (False, True):
        ref_o, ref_l = qa.fwd(tq, tk, tv, causal=causal)
        for _ in range(2):
            o, l = qa.fwd(tq, tk, tv, causal=causal)
            torch.cuda.synchronize()
            assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
            assert torch.equal(l.view(torch.int32), ref_l.view(torch.int32))
