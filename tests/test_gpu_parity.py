"""GPU parity: the gfx950 kernels through the C ABI against the fp64 oracle.

Every case draws seeded inputs, runs ``qm_attn_fwd`` on the GPU and compares
element by element with the oracle on the same 16-bit inputs (gate in
``tests/gpu_util.py``; every case prints its raw max-abs errors).  Every
quoted workload is compared in full, the long ones (N = 2048, 8192, 32768) in
the launch configuration that ``bench.py`` times, with the oracle spread over
processes; sampled rows that the oracle computes one by one, and properties
that hold at any size, are cheap extra checks.
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


def run_gpu(qa, q, k, v, dtype, scale, causal):
    import torch
    tq, tk, tv = (to_device(x, dtype) for x in (q, k, v))
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=scale)
    torch.cuda.synchronize()
    return to_host64(o), to_host64(lse)


def full_case(qa, q, k, v, dtype, scale, causal, what):
    _say(f"case {what}: shape={q.shape} dtype={dtype} scale={scale} causal={causal}")
    Og, lg = run_gpu(qa, q, k, v, dtype, scale, causal)
    Or, lr = attention_fp64(q, k, v, scale, causal, dtype)
    return check_close(Og, lg, Or, lr, dtype, what)


# ---------------------------------------------------------------- workloads
@pytest.mark.parametrize("name", ["mha_b1_h2_n128_d64_f16", "mha_b8_h16_n1024_d64_f16"])
def test_small_workloads_full(qa, name):
    w = si.WORKLOADS[name]
    q, k, v = w.inputs()
    for causal in (False, True):
        full_case(qa, q, k, v, w.dtype, w.scale, causal, f"{name} causal={causal}")


_INPUTS = {}


def _inputs(name):
    """Seeded inputs of a named workload, drawn once per module."""
    if name not in _INPUTS:
        _say(f"drawing the inputs of {name}")
        _INPUTS.clear()
        _INPUTS[name] = si.WORKLOADS[name].inputs()
    return _INPUTS[name]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,causal", [
    ("mha_b4_h32_n2048_d128_f16_causal", True),
    ("mha_b2_h32_n8192_d128_bf16", False),
    ("mha_b2_h32_n8192_d128_bf16", True),
    ("mha_b1_h32_n32768_d128_bf16_causal_qk2", True),
])
def test_workloads_every_element(qa, name, causal):
    """The quoted long workloads in the launch configuration the benchmark
    times, every output element compared with the oracle (all heads, the
    oracle spread over processes; ``tests/oracle_pool.py``)."""
    import torch
    from tests import oracle_pool
    w = si.WORKLOADS[name]
    q, k, v = _inputs(name)
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    _say(f"case {name} causal={causal}: running (full comparison)")
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    bits, L = oracle_pool.gpu_bits(o), lse.cpu().numpy()
    del o, lse, tq, tk, tv
    oracle_pool.full_compare(q, k, v, bits, L, w.scale, causal, w.dtype,
                             f"{name} causal={causal}")


def _sample_rows(w, n, seed):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 31, 32, 63, 64, 127, 128, 129, w.N // 2, w.N - 129, w.N - 128, w.N - 2, w.N - 1]
    rows = []
    for t in range(n):
        b = int(rng.integers(w.B))
        h = int(rng.integers(w.H))
        i = fixed[t] if t < len(fixed) else int(rng.integers(w.N))
        rows.append((b, h, i))
    return rows


@pytest.mark.parametrize("name,causal", [
    ("mha_b2_h32_n8192_d128_bf16", False),
    ("mha_b2_h32_n8192_d128_bf16", True),
    ("mha_b1_h32_n32768_d128_bf16_causal_qk2", True),
])
def test_long_workloads_sampled(qa, name, causal):
    import torch
    w = si.WORKLOADS[name]
    q, k, v = _inputs(name)
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    _say(f"case {name} causal={causal}: running")
    o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale)
    torch.cuda.synchronize()
    # properties at full size: finite, and every output a convex combination of V rows
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    vmax = float(tv.abs().amax(dim=2).float().max())
    assert float(o.abs().float().max()) <= vmax * (1 + 2 ** -7)
    rows = _sample_rows(w, 128, seed=2)
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    Og = to_host64(o[ix])
    lg = to_host64(lse[ix])
    _say(f"case {name} causal={causal}: oracle on {len(rows)} rows")
    Or, lr = attention_rows_fp64(q, k, v, w.scale, causal, w.dtype, rows)
    check_close(Og, lg, Or, lr, w.dtype, f"{name} causal={causal} sampled rows")
    if causal and name.startswith("mha_b2"):
        # the last causal row sees every key: it equals the unmasked run bit for bit
        o2, l2 = qa.fwd(tq, tk, tv, causal=False, scale=w.scale)
        torch.cuda.synchronize()
        assert torch.equal(o[:, :, -1], o2[:, :, -1])
        assert torch.equal(lse[:, :, -1], l2[:, :, -1])


@pytest.mark.parametrize("name", sorted(si.GRID))
def test_paper_grid_sampled(qa, name):
    """Every shape of the paper's benchmark grid, both masks, on sampled rows."""
    import torch
    w = si.GRID[name]
    _say(f"case {name}: drawing inputs")
    q, k, v = w.inputs()
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    rows = _sample_rows(w, 24, seed=5)
    ix = tuple(torch.tensor(np.array(rows).T).cuda())
    for causal in w.causal:
        _say(f"case {name} causal={causal}")
        o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=w.scale)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        Or, lr = attention_rows_fp64(q, k, v, w.scale, causal, w.dtype, rows)
        check_close(to_host64(o[ix]), to_host64(lse[ix]), Or, lr, w.dtype,
                    f"{name} causal={causal} sampled rows")


# ---------------------------------------------------------------- edge shapes
EDGE_N = [1, 2, 17, 63, 64, 65, 127, 128, 129, 255, 1000]


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("N", EDGE_N)
def test_edge_shapes(qa, N, dtype, d):
    q, k, v = si.make_qkv(2, 3, N, d, dtype, seed=N * 7 + d)
    for causal in (False, True):
        full_case(qa, q, k, v, dtype, si.default_scale(d), causal,
                  f"edge N={N} d={d} {dtype} causal={causal}")


# ---------------------------------------------------------------- special inputs
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("d", [64, 128])
def test_special_inputs(qa, dtype, d):
    B, H, N = 1, 2, 300
    q, k, v = si.make_qkv(B, H, N, d, dtype, seed=5 + d)
    zero = np.zeros_like(q)
    const_v = np.broadcast_to(v[:, :, :1], v.shape).copy()
    # sharp rows: query i is 8x key (i*7 mod N), an exact power-of-two multiple
    perm = (np.arange(N) * 7) % N
    if dtype == "f16":
        sharp_q = (k[:, :, perm].astype(np.float32) * 8).astype(np.float16)
    else:
        sharp_q = si.f32_to_bf16_bits(
            (k[:, :, perm].astype(np.uint32) << 16).view(np.float32) * 8)
    cases = [
        ("zero Q", zero, k, v, si.default_scale(d)),
        ("scale 0", q, k, v, 0.0),
        ("scale 1e-40", q, k, v, 1e-40),
        ("negative scale", q, k, v, -0.37),
        ("large scores", q, k, v, 5.0),          # |score| up to ~60
        ("constant V", q, k, const_v, si.default_scale(d)),
        ("one-hot rows", sharp_q, k, v, si.default_scale(d)),
    ]
    for what, qq, kk, vv, scale in cases:
        for causal in (False, True):
            full_case(qa, qq, kk, vv, dtype, scale, causal,
                      f"{what} d={d} {dtype} causal={causal}")


def test_zero_query_closed_form(qa):
    """Q = 0: O is the (prefix) mean of V and lse = ln(#visible keys), directly."""
    B, H, N, d = 1, 2, 200, 64
    _, k, v = si.make_qkv(B, H, N, d, "f16", seed=3)
    q = np.zeros_like(k)
    vf = v.astype(np.float64)
    for causal in (False, True):
        Og, lg = run_gpu(qa, q, k, v, "f16", 0.125, causal)
        n = np.arange(1, N + 1) if causal else np.full(N, N)
        mean = np.cumsum(vf, axis=2) / n[:, None] if causal else np.broadcast_to(
            vf.mean(axis=2, keepdims=True), vf.shape)
        check_close(Og, lg, mean, np.broadcast_to(np.log(n), lg.shape), "f16",
                    f"zero-Q closed form causal={causal}")


# ---------------------------------------------------------------- structure
def test_head_slices_are_independent(qa):
    """A (batch, head) slice run alone equals that slice of the batched run, bitwise."""
    import torch
    q, k, v = si.make_qkv(2, 3, 333, 128, "bf16", seed=9)
    tq, tk, tv = (to_device(x, "bf16") for x in (q, k, v))
    for causal in (False, True):
        o, lse = qa.fwd(tq, tk, tv, causal=causal)
        for b, h in [(0, 0), (1, 2), (0, 1)]:
            sl = (slice(b, b + 1), slice(h, h + 1))
            o1, l1 = qa.fwd(tq[sl].contiguous(), tk[sl].contiguous(), tv[sl].contiguous(),
                            causal=causal)
            torch.cuda.synchronize()
            assert torch.equal(o1, o[sl]) and torch.equal(l1, lse[sl])


def test_bit_stable_across_runs_and_streams(qa):
    import torch
    q, k, v = si.make_qkv(2, 4, 1111, 64, "f16", seed=10)
    tq, tk, tv = (to_device(x, "f16") for x in (q, k, v))
    for causal in (False, True):
        ref_o, ref_l = qa.fwd(tq, tk, tv, causal=causal)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        for rep in range(3):
            with torch.cuda.stream(s if rep == 2 else torch.cuda.current_stream()):
                o, l = qa.fwd(tq, tk, tv, causal=causal)
            torch.cuda.synchronize()
            assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
            assert torch.equal(l.view(torch.int32), ref_l.view(torch.int32))


def test_every_output_written_and_nothing_else(qa):
    """NaN-poisoned outputs are fully overwritten; guard zones around them are untouched."""
    import torch
    B, H, N, d = 2, 2, 197, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=11)
    tq, tk, tv = (to_device(x, "bf16") for x in (q, k, v))
    G = 256   # guard elements on each side (keeps 16-byte alignment)
    for causal in (False, True):
        obuf = torch.full((B * H * N * d + 2 * G,), float("nan"), dtype=torch.bfloat16,
                          device="cuda")
        lbuf = torch.full((B * H * N + 2 * G,), float("nan"), dtype=torch.float32, device="cuda")
        obuf[:G] = 7.0
        obuf[-G:] = 7.0
        lbuf[:G] = 7.0
        lbuf[-G:] = 7.0
        o = obuf[G:G + B * H * N * d].view(B, H, N, d)
        lse = lbuf[G:G + B * H * N].view(B, H, N)
        qa.fwd(tq, tk, tv, causal=causal, out=o, lse=lse)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        assert bool((obuf[:G] == 7.0).all()) and bool((obuf[-G:] == 7.0).all())
        assert bool((lbuf[:G] == 7.0).all()) and bool((lbuf[-G:] == 7.0).all())
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), causal, "bf16")
        check_close(to_host64(o), to_host64(lse), Or, lr, "bf16", f"poisoned causal={causal}")


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f16", 64)])
def test_inputs_read_only_within_bounds(qa, dtype, d):
    """Rows past the end of the sequence read as zeros: NaN placed right after the
    last head of Q, K and V never reaches the outputs.  The guard is longer than
    one key block, so every read stays inside the allocation either way."""
    import torch
    B, H, N = 2, 2, 197          # 197 = 3 * 64 + 5: the last key block has 59 missing rows
    q, k, v = si.make_qkv(B, H, N, d, dtype, seed=12)
    G = 2 * 64 * d
    n = B * H * N * d
    bufs = []
    for x in (q, k, v):
        t = to_device(x, dtype).reshape(-1)
        buf = torch.full((n + G,), float("nan"), dtype=t.dtype, device="cuda")
        buf[:n] = t
        bufs.append(buf)
    tq, tk, tv = (b[:n].view(B, H, N, d) for b in bufs)
    for causal in (False, True):
        _say(f"case guarded inputs: dtype={dtype} d={d} causal={causal}")
        o, lse = qa.fwd(tq, tk, tv, causal=causal)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), causal, dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, dtype, f"guarded inputs causal={causal}")


def test_invalid_arguments_enqueue_nothing(qa):
    import torch
    x = torch.zeros(1, 1, 64, 96, dtype=torch.float16, device="cuda")
    with pytest.raises(qa.QmAttnError) as e:
        qa.fwd(x, x, x)
    assert e.value.status == qa.QM_ERR_HEADDIM
    y = torch.zeros(1, 1, 64, 64, dtype=torch.float16, device="cuda")
    with pytest.raises(qa.QmAttnError) as e:
        qa.fwd(y, y, y, out=y)
    assert e.value.status == qa.QM_ERR_ALIAS


def test_non_finite_inputs_stay_in_the_outputs_that_read_them(qa):
    """NaN in one query row, and infinity in one key of one key/value head:
    every other output matches the oracle on the same inputs, and the kernel
    completes."""
    import torch
    B, H, Hkv, N, d = 2, 4, 2, 300, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=130, Hkv=Hkv)
    q = q.copy()
    k = k.copy()
    q[1, 3, 17, 5] = 0x7FC0          # bf16 NaN in query row 17 of (batch 1, head 3)
    k[0, 1, 200, 9] = 0x7F80         # bf16 +inf in key 200 of (batch 0, kv head 1)
    scale = si.default_scale(d)
    clean = np.ones((B, H, N), dtype=bool)
    clean[1, 3, 17] = False
    clean[0, 2:4] = False            # query heads 2 and 3 read kv head 1
    qc, kc = q.copy(), k.copy()
    qc[1, 3, 17, 5] = 0
    kc[0, 1, 200, 9] = 0
    for causal in (False, True):
        o, lse = qa.fwd(*(to_device(x, "bf16") for x in (q, k, v)), causal=causal, scale=scale)
        torch.cuda.synchronize()
        O, L = to_host64(o), to_host64(lse)
        Or, lr = attention_fp64(qc, kc, v, scale, causal, "bf16")
        check_close(O[clean], L[clean], Or[clean], lr[clean], "bf16",
                    f"finite outputs next to non-finite inputs causal={causal}")


def test_bench_workload_bit_stable_under_sustained_load(qa):
    """The benchmark workload (B = 2, H = 32, N = 8192, d = 128, bf16), both
    masks, launched back to back 40 times each as the benchmark does: every
    launch gives the bytes of the first (the clock moves under sustained load;
    the results must not)."""
    import torch
    w = si.WORKLOADS["mha_b2_h32_n8192_d128_bf16"]
    tq, tk, tv = (to_device(x, "bf16") for x in w.inputs())
    refs = [qa.fwd(tq, tk, tv, causal=c, scale=w.scale) for c in (False, True)]
    torch.cuda.synchronize()
    outs = [(torch.empty_like(o), torch.empty_like(l)) for o, l in refs]
    mismatches = torch.zeros(2, dtype=torch.int64, device="cuda")
    for _ in range(40):
        for m, c in enumerate((False, True)):
            qa.fwd(tq, tk, tv, causal=c, scale=w.scale, out=outs[m][0], lse=outs[m][1])
            mismatches[m] += (outs[m][0].view(torch.int16) != refs[m][0].view(torch.int16)).sum()
            mismatches[m] += (outs[m][1].view(torch.int32) != refs[m][1].view(torch.int32)).sum()
    torch.cuda.synchronize()
    assert mismatches.tolist() == [0, 0]
