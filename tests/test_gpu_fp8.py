"""GPU parity for the FP8 forward (``qm_attn_fwd_fp8``, and
``qm_attn_fwd_fp8_layout`` for fewer key/value heads and the [B][N][H][d]
layout): OCP E4M3 inputs with per-tensor scale factors, bf16 output, head
dimension 128.

Two roundings separate the kernel from the exact definition on general
inputs.

* P is rounded to E4M3 for the P.V product: relative error at most 2^-4 for a
  normal value, absolute at most 2^-10 (half the subnormal spacing 2^-9) in
  units of the largest weight, since the weights are formed against a running
  maximum no larger than the row's true maximum.
* The FP8 matrix-core instruction sums its 64 products in groups of 8
  consecutive k: within a group every product is truncated toward zero to a
  multiple of 2^(E - 13), E the exponent of the group's largest product, and
  the group sums enter the fp32 accumulator (measured on gfx950 with one-hot
  operands).  A group of 8 thus loses less than 7 x 2^-13 of its largest
  product.  On the scores this is an absolute error of at most
  Delta_i = 7 x 2^-13 |scale q_scale k_scale| max_j sum_c |q_ic k_jc| (plus
  fp32 rounding), which moves each normalised weight by a factor within
  exp(+-2 Delta_i); on P.V it is at most 7 x 2^-13 of sum_j P_ij |v_jc|.

Per output element (row i, column c), with P the exact softmax weights and v
the real (scaled) values:

    |O - O_ref| <= ((1 + 2^-4) e^(2 Delta_i) (1 + 7 x 2^-13) - 1) sum_j P_ij |v_jc|
                   + 2^-10 e^(2 Delta_i) max_j P_ij sum_j |v_jc|
                   + half a bf16 ulp + fp32 summation terms.

That bound is loose for a layout test, so most cases use inputs on which no
rounding happens: integer scores in [-4, 4] and a combined softmax scale of
ln 2 make every weight a power of two between 2^-8 and 2^8 (relative to any
maximum the kernel may hold), all exact in E4M3; Q.K products are small
integers, which no group truncates; with V in one binade the P.V products of
a group span less than 2^10, so their truncation drops nothing either.
There the kernel must match the oracle to fp32 summation error and the bf16
output rounding.  With V over all E4M3 codes only the P.V group truncation
is added.  Independently of the oracle, the FP8 kernel must agree with the
bf16 kernel on the same real values when neither rounds.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import seeded_inputs as si
from oracle import (attention_fp64, attention_rows_fp64, decode_fp64, scores_fp64,
                    softmax_rows_fp64)
from tests import oracle_pool
from tests.fp8_gate import GROUP_TRUNC, rounding_bound
from tests.fp8_gate import summation as _summation
from tests.gpu_util import assert_stats, compare, half_ulp, to_host64

pytestmark = pytest.mark.gpu

LN2 = math.log(2.0)


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


def _codes(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda().view(torch.float8_e4m3fn)


def _run(qa, q8, k8, v8, scales, causal, scale):
    import torch
    o, lse = qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=causal, scale=scale)
    torch.cuda.synchronize()
    return to_host64(o), to_host64(lse)


def _gate(O, lse, Or, lr, bound, what):
    """Per-element bound on |O - Or|, lse within 1e-3; prints the raw errors."""
    st = compare(O, lse, Or, lr, "bf16", bound=bound)
    assert_stats(st, "bf16", what)
    return st["max_err"], st["max_lse_err"]


def _tight_case(qa, q8, k8, v8, scales, causal, scale, what, pv_trunc=False):
    """Exact-weight inputs: the oracle's value up to fp32 summation and the
    bf16 output rounding (plus, with ``pv_trunc``, the P.V group truncation)."""
    _say(f"case {what}: shape={q8.shape} scales={scales} scale={scale} causal={causal}")
    O, lse = _run(qa, q8, k8, v8, scales, causal, scale)
    Or, lr = attention_fp64(q8, k8, v8, scale, causal, "e4m3", descale=scales)
    PV, _ = attention_fp64(q8, k8, v8 & 0x7F, scale, causal, "e4m3", descale=scales)
    N = q8.shape[2]
    rel = _summation(N) + (GROUP_TRUNC if pv_trunc else 0.0)
    bound = half_ulp(Or, "bf16") + rel * PV
    return _gate(O, lse, Or, lr, bound, what)


# -------------------------------------------------- exact-rounding inputs
@pytest.mark.parametrize("scales,scale", [
    ((0.5, 2.0, 0.0123), LN2),            # q_scale * k_scale = 1
    ((0.25, 2.0, 1.0), 2 * LN2),          # q_scale * k_scale = 1/2
    ((1.0, 1.0, 3.5), -LN2),              # negative scale: the kernel flips Q's signs
])
def test_dyadic_inputs_full(qa, scales, scale):
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, 3, 333, 128, seed=11, v_binade=True)
    for causal in (False, True):
        _tight_case(qa, q8, k8, v8, scales, causal, scale, f"dyadic scales={scales}")


def test_dyadic_inputs_all_value_codes(qa):
    """Every E4M3 code in V (subnormals, both zeros, 448): the decode of V is
    exact, only the matrix core's in-group truncation of P.V is allowed."""
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, 3, 333, 128, seed=11)
    for causal in (False, True):
        _tight_case(qa, q8, k8, v8, (0.5, 2.0, 0.0123), causal, LN2, "dyadic, all V codes",
                    pv_trunc=True)


@pytest.mark.parametrize("N", [1, 2, 63, 64, 65, 129, 255, 1000, 2111])
def test_dyadic_edge_lengths(qa, N):
    q8, k8, v8 = si.make_qkv_fp8_dyadic(1, 2, N, 128, seed=N, v_binade=True)
    for causal in (False, True):
        _tight_case(qa, q8, k8, v8, (1.0, 1.0, 0.01), causal, LN2, f"dyadic N={N}")


def test_negligible_scores_give_uniform_weights(qa):
    """A combined score scale too small to change any score: every visible key
    weighs the same (the kernel zeroes Q; the oracle's scores are ~1e-60)."""
    q8, k8, v8 = si.make_qkv_fp8_dyadic(1, 2, 300, 128, seed=5, v_binade=True)
    for causal in (False, True):
        _tight_case(qa, q8, k8, v8, (1e-30, 1e-30, 0.25), causal, 0.088,
                    f"negligible scores causal={causal}")


def test_fp8_agrees_with_bf16_kernel(qa):
    """Same real values through both kernels: Q = +-1/2 and K = 2 x integers
    (exact in bf16), V = 2^-6 x one-binade E4M3 values (exact in bf16), and
    power-of-two weights that neither kernel rounds.  Only the fp32 summation
    order and the output rounding may differ."""
    import torch
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, 4, 700, 128, seed=21, v_binade=True)
    scales = (0.5, 2.0, 2.0 ** -6)
    for causal in (False, True):
        _say(f"case fp8 vs bf16 causal={causal}")
        O8, l8 = _run(qa, q8, k8, v8, scales, causal, LN2)
        real = [torch.from_numpy(decode_fp64(x, "e4m3") * s).to(torch.bfloat16).cuda()
                for x, s in zip((q8, k8, v8), scales)]
        for t, x, s in zip(real, (q8, k8, v8), scales):
            assert np.array_equal(t.double().cpu().numpy(), decode_fp64(x, "e4m3") * s)
        o16, l16 = qa.fwd(*real, causal=causal, scale=LN2)
        torch.cuda.synchronize()
        O16, L16 = to_host64(o16), to_host64(l16)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        bound = (np.maximum(half_ulp(O8, "bf16"), half_ulp(O16, "bf16")) * 2
                 + 2 * _summation(700) * PV)
        _gate(O8, l8, O16, L16, bound, f"fp8 vs bf16 causal={causal}")


# -------------------------------------------------- general FP8 inputs
def _rounding_bound(q8, k8, v8, scales, scale, causal, rows, O, Or):
    """The general-input bound (``tests/fp8_gate.py``) for the given (b, h, i)
    rows, from the oracle's own scores and weights; O is unused (the bound
    depends on the oracle's values only)."""
    group = q8.shape[1] // k8.shape[1]   # query heads per key/value head
    bound = np.empty_like(Or)
    by_head = {}
    for idx, (b, h, i) in enumerate(rows):
        by_head.setdefault((b, h), []).append((idx, i))
    for (b, h), items in by_head.items():
        idxs = [t for t, _ in items]
        rr = np.array([i for _, i in items])
        bound[idxs] = rounding_bound(q8[b, h, rr], k8[b, h // group], v8[b, h // group],
                                     scales, scale, causal, rr, Or[idxs])
    return bound


def test_small_fp8_workload_full(qa):
    w = si.WORKLOADS["fp8_b2_h3_n333_d128"]
    q8, k8, v8, scales = w.fp8_inputs()
    rows = [(b, h, i) for b in range(w.B) for h in range(w.H) for i in range(w.N)]
    for causal in w.causal:
        _say(f"case {w.name} causal={causal}")
        O, lse = _run(qa, q8, k8, v8, scales, causal, w.scale)
        Or, lr = attention_fp64(q8, k8, v8, w.scale, causal, "e4m3", descale=scales)
        Of, Orf = O.reshape(-1, w.d), Or.reshape(-1, w.d)
        bound = _rounding_bound(q8, k8, v8, scales, w.scale, causal, rows, Of, Orf)
        err, _ = _gate(Of, lse.ravel(), Orf, lr.ravel(), bound, f"{w.name} causal={causal}")
        # the bound is worst case; rounding errors of independent weights mostly
        # cancel, so the typical error sits far below it
        rms = float(np.sqrt(np.mean((Of - Orf) ** 2)))
        assert rms < 0.1 * float(np.sqrt(np.mean(bound ** 2))), rms


def _sample_rows(w, n, seed):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 63, 64, 255, 256, w.N // 2, w.N - 257, w.N - 2, w.N - 1]
    return [(int(rng.integers(w.B)), int(rng.integers(w.H)),
             fixed[t] if t < len(fixed) else int(rng.integers(w.N))) for t in range(n)]


@pytest.fixture(scope="module")
def long_inputs():
    w = si.WORKLOADS["fp8_b2_h32_n8192_d128"]
    _say(f"drawing the inputs of {w.name}")
    return w, w.fp8_inputs()


@pytest.mark.parametrize("causal", [False, True])
def test_long_fp8_workload_sampled(qa, long_inputs, causal):
    """The FP8 benchmark workload (B = 2, H = 32, N = 8192, d = 128) in the
    launch configuration the benchmark times, on sampled rows."""
    import torch
    w, (q8, k8, v8, scales) = long_inputs
    tq, tk, tv = _codes(q8), _codes(k8), _codes(v8)
    _say(f"case {w.name} causal={causal}: running")
    o, lse = qa.fwd_fp8(tq, tk, tv, scales, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    vmax = 448.0 * float(np.float32(scales[2]))
    # a convex combination of the values, up to the weights' E4M3 rounding
    assert float(o.abs().float().max()) <= vmax * 1.125
    # the inputs are read only
    assert torch.equal(tq.view(torch.uint8).cpu(), torch.from_numpy(q8))
    assert torch.equal(tv.view(torch.uint8).cpu(), torch.from_numpy(v8))
    rows = sorted(_sample_rows(w, 96, seed=8 + causal))
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    O, L = to_host64(o[ix]), to_host64(lse[ix])
    _say(f"case {w.name} causal={causal}: oracle on {len(rows)} rows")
    Or, lr = attention_rows_fp64(q8, k8, v8, w.scale, causal, "e4m3", rows, descale=scales)
    bound = _rounding_bound(q8, k8, v8, scales, w.scale, causal, rows, O, Or)
    _gate(O, L, Or, lr, bound, f"{w.name} causal={causal} sampled rows")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("causal", [False, True])
def test_long_fp8_workload_full(qa, long_inputs, causal):
    """The FP8 benchmark workload in the launch configuration the benchmark
    times, every output element of all 64 heads under the rounding bound (the
    oracle spread over processes)."""
    import torch
    w, (q8, k8, v8, scales) = long_inputs
    _say(f"case {w.name} causal={causal}: running (full comparison)")
    o, lse = qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    bits, L = oracle_pool.gpu_bits(o), lse.cpu().numpy()
    del o, lse
    oracle_pool.full_compare(q8, k8, v8, bits, L, w.scale, causal, "e4m3",
                             f"{w.name} causal={causal}", descale=scales)


@pytest.mark.parametrize("name", sorted(si.GRID_FP8))
def test_fp8_paper_grid_sampled(qa, name):
    """The paper's FP8 table configuration (16k tokens per batch, hidden 2048,
    d = 128, causal) at every sequence length, on sampled rows."""
    import torch
    w = si.GRID_FP8[name]
    _say(f"case {w.name}: drawing inputs")
    q8, k8, v8, scales = w.fp8_inputs()
    _say(f"case {w.name}: running")
    o, lse = qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    rows = sorted(_sample_rows(w, 24, seed=w.N))
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    O, L = to_host64(o[ix]), to_host64(lse[ix])
    Or, lr = attention_rows_fp64(q8, k8, v8, w.scale, True, "e4m3", rows, descale=scales)
    bound = _rounding_bound(q8, k8, v8, scales, w.scale, True, rows, O, Or)
    _gate(O, L, Or, lr, bound, f"{w.name} sampled rows")


# -------------------------------------------------- memory safety, determinism
def test_fp8_outputs_written_and_nothing_else(qa):
    """NaN-poisoned bf16 outputs are fully overwritten (the output is two bytes
    per element while the inputs are one); guard zones around o and lse stay
    untouched."""
    import torch
    B, H, N, d = 2, 2, 197, 128
    q8, k8, v8 = si.make_qkv_fp8_dyadic(B, H, N, d, seed=31, v_binade=True)
    scales = (1.0, 1.0, 0.05)
    G = 256
    for causal in (False, True):
        obuf = torch.full((B * H * N * d + 2 * G,), float("nan"), dtype=torch.bfloat16,
                          device="cuda")
        lbuf = torch.full((B * H * N + 2 * G,), float("nan"), dtype=torch.float32, device="cuda")
        for buf in (obuf, lbuf):
            buf[:G] = 7.0
            buf[-G:] = 7.0
        o = obuf[G:G + B * H * N * d].view(B, H, N, d)
        lse = lbuf[G:G + B * H * N].view(B, H, N)
        qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=causal, scale=LN2,
                   out=o, lse=lse)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        for buf in (obuf, lbuf):
            assert bool((buf[:G] == 7.0).all()) and bool((buf[-G:] == 7.0).all())
        Or, lr = attention_fp64(q8, k8, v8, LN2, causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        O, L = to_host64(o), to_host64(lse)
        bound = half_ulp(Or, "bf16") + _summation(N) * PV
        _gate(O, L, Or, lr, bound, f"poisoned FP8 outputs causal={causal}")


def test_fp8_inputs_read_only_within_bounds(qa):
    """NaN codes right after the last head of Q, K and V never reach the
    outputs: rows past the end of the sequence read as zeros."""
    import torch
    B, H, N, d = 2, 2, 197, 128
    q8, k8, v8 = si.make_qkv_fp8_dyadic(B, H, N, d, seed=32, v_binade=True)
    n = B * H * N * d
    G = 2 * 64 * d
    views = []
    for x in (q8, k8, v8):
        buf = torch.full((n + G,), 0x7F, dtype=torch.uint8, device="cuda")   # E4M3 NaN
        buf[:n] = torch.from_numpy(x.reshape(-1)).cuda()
        views.append(buf[:n].view(B, H, N, d).view(torch.float8_e4m3fn))
    scales = (1.0, 1.0, 0.05)
    for causal in (False, True):
        _say(f"case guarded FP8 inputs causal={causal}")
        o, lse = qa.fwd_fp8(*views, scales, causal=causal, scale=LN2)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        Or, lr = attention_fp64(q8, k8, v8, LN2, causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        O, L = to_host64(o), to_host64(lse)
        bound = half_ulp(Or, "bf16") + _summation(N) * PV
        _gate(O, L, Or, lr, bound, f"guarded FP8 inputs causal={causal}")


def test_fp8_bit_stable_across_runs_and_streams(qa):
    import torch
    w = si.WORKLOADS["fp8_b2_h3_n333_d128"]
    q8, k8, v8, scales = w.fp8_inputs()
    tq, tk, tv = _codes(q8), _codes(k8), _codes(v8)
    for causal in (False, True):
        ref_o, ref_l = qa.fwd_fp8(tq, tk, tv, scales, causal=causal)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        for rep in range(3):
            with torch.cuda.stream(s if rep == 2 else torch.cuda.current_stream()):
                o, l = qa.fwd_fp8(tq, tk, tv, scales, causal=causal)
            torch.cuda.synchronize()
            assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
            assert torch.equal(l.view(torch.int32), ref_l.view(torch.int32))


@pytest.mark.parametrize("N", [1, 65, 1000])
def test_fp8_general_inputs_edge_lengths(qa, N):
    """General FP8 inputs (normal draws scaled to the E4M3 range) at ragged
    lengths, compared in full under the rounding bound."""
    q8, k8, v8, scales = si.make_qkv_fp8(2, 3, N, 128, seed=50 + N)
    scale = si.default_scale(128)
    rows = [(b, h, i) for b in range(2) for h in range(3) for i in range(N)]
    for causal in (False, True):
        _say(f"case FP8 general inputs N={N} causal={causal}")
        O, lse = _run(qa, q8, k8, v8, scales, causal, scale)
        Or, lr = attention_fp64(q8, k8, v8, scale, causal, "e4m3", descale=scales)
        Of, Orf = O.reshape(-1, 128), Or.reshape(-1, 128)
        bound = _rounding_bound(q8, k8, v8, scales, scale, causal, rows, Of, Orf)
        _gate(Of, lse.ravel(), Orf, lr.ravel(), bound, f"FP8 general N={N} causal={causal}")


# -------------------------------------------------- grouped-query heads, [B][N][H][d]
def _bnhd(x):
    """[B][heads][N][d] array -> contiguous [B][N][heads][d]."""
    return np.ascontiguousarray(np.swapaxes(x, 1, 2))


def _run_any(qa, q8, k8, v8, scales, causal, scale, layout):
    """fwd_fp8 on [B][H][N][d] codes stored in ``layout``; returns the device
    outputs with o in [B][H][N][d] order."""
    import torch
    lay = _bnhd if layout == "bnhd" else (lambda x: x)
    o, lse = qa.fwd_fp8(*(_codes(lay(x)) for x in (q8, k8, v8)), scales, causal=causal,
                        scale=scale, layout=layout)
    torch.cuda.synchronize()
    if layout == "bnhd":
        o = o.transpose(1, 2).contiguous()
    return o, lse


def _same_as_multi_head(qa, o, lse, q8, k8, v8, scales, causal, scale):
    """Byte-identical to the multi-head [B][H][N][d] call with each key/value
    head repeated for its query heads (same arithmetic, other addresses)."""
    import torch
    g = q8.shape[1] // k8.shape[1]
    ob, lb = _run_any(qa, q8, np.repeat(k8, g, axis=1), np.repeat(v8, g, axis=1), scales,
                      causal, scale, "bhnd")
    assert torch.equal(o.view(torch.int16), ob.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lb.view(torch.int32))


@pytest.mark.parametrize("layout", ["bhnd", "bnhd"])
@pytest.mark.parametrize("H,Hkv,N", [(6, 2, 333), (4, 1, 65), (3, 3, 1000), (8, 2, 1)])
def test_fp8_grouped_heads_and_layouts_dyadic(qa, H, Hkv, N, layout):
    """Exact-weight inputs with H query and Hkv key/value heads in either
    layout: the oracle's value up to fp32 summation and the bf16 rounding."""
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, H, N, 128, seed=70 + H + N, v_binade=True, Hkv=Hkv)
    scales = (0.5, 2.0, 0.0123)
    for causal in (False, True):
        what = f"FP8 {layout} H={H} Hkv={Hkv} N={N} causal={causal}"
        _say(f"case {what}")
        o, lse = _run_any(qa, q8, k8, v8, scales, causal, LN2, layout)
        O, L = to_host64(o), to_host64(lse)
        Or, lr = attention_fp64(q8, k8, v8, LN2, causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        bound = half_ulp(Or, "bf16") + _summation(N) * PV
        _gate(O, L, Or, lr, bound, what)
        _same_as_multi_head(qa, o, lse, q8, k8, v8, scales, causal, LN2)


@pytest.mark.parametrize("layout", ["bhnd", "bnhd"])
def test_fp8_grouped_workload_full(qa, layout):
    """General FP8 inputs, 6 query / 2 key-value heads, N = 555, in full under
    the rounding bound."""
    w = si.WORKLOADS["fp8_gqa_b2_h6_kv2_n555_d128"]
    q8, k8, v8, scales = w.fp8_inputs()
    assert k8.shape == (w.B, w.kv_heads, w.N, w.d)
    rows = [(b, h, i) for b in range(w.B) for h in range(w.H) for i in range(w.N)]
    for causal in w.causal:
        what = f"{w.name} {layout} causal={causal}"
        _say(f"case {what}")
        o, lse = _run_any(qa, q8, k8, v8, scales, causal, w.scale, layout)
        O, L = to_host64(o), to_host64(lse)
        Or, lr = attention_fp64(q8, k8, v8, w.scale, causal, "e4m3", descale=scales)
        Of, Orf = O.reshape(-1, w.d), Or.reshape(-1, w.d)
        bound = _rounding_bound(q8, k8, v8, scales, w.scale, causal, rows, Of, Orf)
        _gate(Of, L.ravel(), Orf, lr.ravel(), bound, what)
        _same_as_multi_head(qa, o, lse, q8, k8, v8, scales, causal, w.scale)


def test_fp8_grouped_long_workload_sampled(qa):
    """64 query / 8 key-value heads, N = 8192, causal, on sampled rows."""
    import torch
    w = si.WORKLOADS["fp8_gqa_b2_h64_kv8_n8192_d128_causal"]
    _say(f"case {w.name}: drawing inputs")
    q8, k8, v8, scales = w.fp8_inputs()
    _say(f"case {w.name}: running")
    o, lse = qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    rows = sorted(_sample_rows(w, 64, seed=71))
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    O, L = to_host64(o[ix]), to_host64(lse[ix])
    Or, lr = attention_rows_fp64(q8, k8, v8, w.scale, True, "e4m3", rows, descale=scales)
    bound = _rounding_bound(q8, k8, v8, scales, w.scale, True, rows, O, Or)
    _gate(O, L, Or, lr, bound, f"{w.name} sampled rows")


@pytest.mark.timeout(900)
def test_fp8_grouped_long_workload_full(qa):
    """64 query / 8 key-value heads, N = 8192, causal: every output element of
    all 128 query heads under the rounding bound."""
    import torch
    w = si.WORKLOADS["fp8_gqa_b2_h64_kv8_n8192_d128_causal"]
    _say(f"case {w.name}: drawing inputs")
    q8, k8, v8, scales = w.fp8_inputs()
    _say(f"case {w.name}: running (full comparison)")
    o, lse = qa.fwd_fp8(_codes(q8), _codes(k8), _codes(v8), scales, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    bits, L = oracle_pool.gpu_bits(o), lse.cpu().numpy()
    del o, lse
    oracle_pool.full_compare(q8, k8, v8, bits, L, w.scale, True, "e4m3", w.name,
                             descale=scales)


@pytest.mark.parametrize("causal", [False, True])
def test_fp8_bnhd_bench_shape_matches_bhnd(qa, long_inputs, causal):
    """The FP8 benchmark shape (B = 2, H = 32, N = 8192) stored [B][N][H][d]:
    byte-identical to the [B][H][N][d] launch, and on sampled rows within
    the rounding bound of the oracle."""
    import torch
    w, (q8, k8, v8, scales) = long_inputs
    _say(f"case {w.name} bnhd causal={causal}")
    o, lse = _run_any(qa, q8, k8, v8, scales, causal, w.scale, "bnhd")
    ob, lb = _run_any(qa, q8, k8, v8, scales, causal, w.scale, "bhnd")
    assert torch.equal(o.view(torch.int16), ob.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), lb.view(torch.int32))
    rows = sorted(_sample_rows(w, 32, seed=72 + causal))
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    O, L = to_host64(o[ix]), to_host64(lse[ix])
    Or, lr = attention_rows_fp64(q8, k8, v8, w.scale, causal, "e4m3", rows, descale=scales)
    bound = _rounding_bound(q8, k8, v8, scales, w.scale, causal, rows, O, Or)
    _gate(O, L, Or, lr, bound, f"{w.name} bnhd causal={causal} sampled rows")


def test_fp8_bnhd_bounds_and_outputs(qa):
    """[B][N][H][d] codes with NaN codes right after each input: rows past the
    end read as zeros although a head's rows are heads x d bytes apart; a
    NaN-poisoned output is fully overwritten and its guard zones stay."""
    import torch
    B, H, Hkv, N, d = 2, 4, 2, 197, 128
    q8, k8, v8 = si.make_qkv_fp8_dyadic(B, H, N, d, seed=73, v_binade=True, Hkv=Hkv)
    views = []
    for x in (q8, k8, v8):
        t = _bnhd(x).reshape(-1)
        buf = torch.full((t.size + 2 * 64 * H * d,), 0x7F, dtype=torch.uint8, device="cuda")
        buf[:t.size] = torch.from_numpy(t).cuda()
        views.append(buf[:t.size].view(B, N, x.shape[1], d).view(torch.float8_e4m3fn))
    scales = (1.0, 1.0, 0.05)
    G = 256
    for causal in (False, True):
        _say(f"case FP8 bnhd guarded causal={causal}")
        obuf = torch.full((B * N * H * d + 2 * G,), float("nan"), dtype=torch.bfloat16,
                          device="cuda")
        obuf[:G] = 7.0
        obuf[-G:] = 7.0
        o = obuf[G:G + B * N * H * d].view(B, N, H, d)
        o, lse = qa.fwd_fp8(*views, scales, causal=causal, scale=LN2, out=o, layout="bnhd")
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        assert bool((obuf[:G] == 7.0).all()) and bool((obuf[-G:] == 7.0).all())
        Or, lr = attention_fp64(q8, k8, v8, LN2, causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, LN2, causal, "e4m3", descale=scales)
        O, L = np.swapaxes(to_host64(o), 1, 2), to_host64(lse)
        bound = half_ulp(Or, "bf16") + _summation(N) * PV
        _gate(O, L, Or, lr, bound, f"FP8 bnhd guarded causal={causal}")
