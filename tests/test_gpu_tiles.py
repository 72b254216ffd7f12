"""The two workgroup sizes (256 query rows with eight wavefronts, 128 rows with
four) give the same bytes: every query row takes the same arithmetic in the
same order whichever tile holds it.  Each case runs with 128-row tiles forced,
256-row tiles forced and the automatic choice, compares the three byte for
byte, and checks the 128-row result against the oracle."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64, attention_rows_fp64
from tests.gpu_util import check_close, half_ulp, to_device, to_host64

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
    yield qa
    qa.set_tile_rows(0)


def _three_ways(qa, call):
    import torch
    res = []
    for rows in (128, 256, 0):
        qa.set_tile_rows(rows)
        o, lse = call()
        torch.cuda.synchronize()
        res.append((o, lse))
    qa.set_tile_rows(0)
    for o, lse in res[1:]:
        assert torch.equal(o.view(torch.int16), res[0][0].view(torch.int16))
        assert torch.equal(lse.view(torch.int32), res[0][1].view(torch.int32))
    return res[0]


@pytest.mark.parametrize("B,H,Hkv,N,d,dtype", [
    (2, 3, 3, 1, 64, "f16"), (2, 3, 3, 65, 128, "bf16"), (1, 4, 2, 300, 64, "bf16"),
    (2, 2, 2, 1000, 128, "f16"), (1, 6, 1, 2049, 128, "bf16"), (1, 2, 2, 3000, 64, "f16"),
])
def test_16bit_tiles_agree(qa, B, H, Hkv, N, d, dtype):
    q, k, v = si.make_qkv(B, H, N, d, dtype, seed=150 + N + d, Hkv=Hkv)
    tq, tk, tv = (to_device(x, dtype) for x in (q, k, v))
    for causal in (False, True):
        _say(f"case tiles B={B} H={H} Hkv={Hkv} N={N} d={d} {dtype} causal={causal}")
        o, lse = _three_ways(qa, lambda: qa.fwd(tq, tk, tv, causal=causal))
        Or, lr = attention_fp64(q, k, v, si.default_scale(d), causal, dtype)
        check_close(to_host64(o), to_host64(lse), Or, lr, dtype,
                    f"128-row tiles N={N} d={d} causal={causal}")


@pytest.mark.parametrize("H,Hkv,N", [(3, 3, 333), (4, 2, 2500)])
def test_fp8_tiles_agree(qa, H, Hkv, N):
    import torch
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, H, N, 128, seed=160 + N, v_binade=True, Hkv=Hkv)
    codes = [torch.from_numpy(x).cuda().view(torch.float8_e4m3fn) for x in (q8, k8, v8)]
    scales = (0.5, 2.0, 0.0123)
    for causal in (False, True):
        _say(f"case FP8 tiles H={H} Hkv={Hkv} N={N} causal={causal}")
        o, lse = _three_ways(qa, lambda: qa.fwd_fp8(*codes, scales, causal=causal,
                                                    scale=math.log(2.0)))
        O, L = to_host64(o), to_host64(lse)
        Or, lr = attention_fp64(q8, k8, v8, math.log(2.0), causal, "e4m3", descale=scales)
        PV, _ = attention_fp64(q8, k8, v8 & 0x7F, math.log(2.0), causal, "e4m3", descale=scales)
        bound = (half_ulp(Or, "bf16")
                 + (2 * (N + 128) * 2.0 ** -24 + 1e-5) * PV)
        assert np.all(np.abs(O - Or) <= bound)
        assert np.max(np.abs(L - lr)) <= 1e-3


def test_bench_shape_tiles_agree(qa):
    """B = 2, H = 32, N = 8192, d = 128, bf16: the automatic choice (256 rows
    here) and forced 128-row tiles give the same bytes at full size."""
    import torch
    w = si.WORKLOADS["mha_b2_h32_n8192_d128_bf16"]
    tq, tk, tv = (to_device(x, "bf16") for x in w.inputs())
    for causal in (False, True):
        _say(f"case bench shape tiles causal={causal}")
        _three_ways(qa, lambda: qa.fwd(tq, tk, tv, causal=causal, scale=w.scale))


def _random_configs(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        d = int(rng.choice([64, 128]))
        H = int(rng.integers(1, 9))
        out.append(dict(B=int(rng.integers(1, 4)), H=H,
                        Hkv=int(rng.choice([x for x in range(1, H + 1) if H % x == 0])),
                        N=int(rng.integers(1, 5000)), d=d,
                        dtype=str(rng.choice(["f16", "bf16"])), causal=bool(rng.integers(2)),
                        seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("c", _random_configs(16, seed=2027), ids=lambda c: (
    f"B{c['B']}H{c['H']}kv{c['Hkv']}N{c['N']}d{c['d']}{c['dtype']}{'c' if c['causal'] else 'u'}"))
def test_random_shapes_tiles_agree(qa, c):
    """Seeded random shapes up to N = 5000, across the automatic choice's
    threshold: both tile sizes give the same bytes, and sampled rows match
    the oracle."""
    _say(f"case random tiles {c}")
    q, k, v = si.make_qkv(c["B"], c["H"], c["N"], c["d"], c["dtype"], seed=c["seed"],
                          Hkv=c["Hkv"])
    tq, tk, tv = (to_device(x, c["dtype"]) for x in (q, k, v))
    o, lse = _three_ways(qa, lambda: qa.fwd(tq, tk, tv, causal=c["causal"]))
    rng = np.random.default_rng(c["seed"])
    rows = [(int(rng.integers(c["B"])), int(rng.integers(c["H"])), int(rng.integers(c["N"])))
            for _ in range(8)] + [(c["B"] - 1, c["H"] - 1, c["N"] - 1)]
    O = np.array([to_host64(o[b, h, i]) for b, h, i in rows])
    L = np.array([float(lse[b, h, i]) for b, h, i in rows])
    Or, lr = attention_rows_fp64(q, k, v, si.default_scale(c["d"]), c["causal"], c["dtype"], rows)
    check_close(O, L, Or, lr, c["dtype"], f"random tiles {c}")
