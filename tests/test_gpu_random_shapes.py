"""Seeded random configurations through every 16-bit entry point, compared in
full with the oracle: batch, heads, key/value heads, length, head dimensions,
type, mask, layout and scale drawn together, so that combinations no
hand-written case names are covered.  FP8 configurations use exact-weight
inputs (integer scores, power-of-two weights) and the tight gate."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64
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
    return qa


def _configs(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        d, dv = [(64, 64), (128, 128), (192, 128)][rng.integers(3)]
        H = int(rng.integers(1, 7))
        Hkv = H if d == 192 else int(rng.choice([x for x in range(1, H + 1) if H % x == 0]))
        out.append(dict(
            B=int(rng.integers(1, 4)), H=H, Hkv=Hkv, N=int(rng.integers(1, 700)), d=d, dv=dv,
            dtype=str(rng.choice(["f16", "bf16"])), causal=bool(rng.integers(2)),
            layout="bhnd" if d == 192 else str(rng.choice(["bhnd", "bnhd"])),
            scale=float(rng.choice([si.default_scale(d), 0.05, -0.3, 1.3])),
            seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("cfg", _configs(32, seed=2025), ids=lambda c: (
    f"B{c['B']}H{c['H']}kv{c['Hkv']}N{c['N']}d{c['d']}v{c['dv']}{c['dtype']}"
    f"{'c' if c['causal'] else 'u'}{c['layout']}"))
def test_random_16bit_configuration(qa, cfg):
    import torch
    c = cfg
    _say(f"case {c}")
    q, k, v = si.make_qkv(c["B"], c["H"], c["N"], c["d"], c["dtype"], seed=c["seed"],
                          Hkv=c["Hkv"], dv=c["dv"])
    bnhd = c["layout"] == "bnhd"
    lay = (lambda x: np.swapaxes(x, 1, 2)) if bnhd else (lambda x: x)
    o, lse = qa.fwd(*(to_device(lay(x), c["dtype"]) for x in (q, k, v)), causal=c["causal"],
                    scale=c["scale"], layout=c["layout"])
    torch.cuda.synchronize()
    O = to_host64(o)
    O = np.swapaxes(O, 1, 2) if bnhd else O
    Or, lr = attention_fp64(q, k, v, c["scale"], c["causal"], c["dtype"])
    check_close(O, to_host64(lse), Or, lr, c["dtype"], f"random {c}")


def _fp8_configs(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        H = int(rng.integers(1, 7))
        out.append(dict(B=int(rng.integers(1, 4)), H=H,
                        Hkv=int(rng.choice([x for x in range(1, H + 1) if H % x == 0])),
                        N=int(rng.integers(1, 700)), causal=bool(rng.integers(2)),
                        layout=str(rng.choice(["bhnd", "bnhd"])),
                        qs=float(rng.choice([0.5, 1.0, 2.0])), vs=float(rng.uniform(0.01, 4.0)),
                        seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("cfg", _fp8_configs(12, seed=2026), ids=lambda c: (
    f"B{c['B']}H{c['H']}kv{c['Hkv']}N{c['N']}{'c' if c['causal'] else 'u'}{c['layout']}"))
def test_random_fp8_configuration(qa, cfg):
    import torch
    c = cfg
    _say(f"case FP8 {c}")
    q8, k8, v8 = si.make_qkv_fp8_dyadic(c["B"], c["H"], c["N"], 128, seed=c["seed"],
                                        v_binade=True, Hkv=c["Hkv"])
    # q_scale * k_scale * scale = ln 2: every weight a power of two, exact in E4M3
    scales = (c["qs"], 1.0 / c["qs"], c["vs"])
    scale = math.log(2.0)
    bnhd = c["layout"] == "bnhd"
    lay = (lambda x: np.swapaxes(x, 1, 2)) if bnhd else (lambda x: x)
    codes = [torch.from_numpy(np.ascontiguousarray(lay(x))).cuda().view(torch.float8_e4m3fn)
             for x in (q8, k8, v8)]
    o, lse = qa.fwd_fp8(*codes, scales, causal=c["causal"], scale=scale, layout=c["layout"])
    torch.cuda.synchronize()
    O = to_host64(o)
    O = np.swapaxes(O, 1, 2) if bnhd else O
    Or, lr = attention_fp64(q8, k8, v8, scale, c["causal"], "e4m3", descale=scales)
    PV, _ = attention_fp64(q8, k8, v8 & 0x7F, scale, c["causal"], "e4m3", descale=scales)
    bound = (half_ulp(Or, "bf16")
             + (2 * (c["N"] + 128) * 2.0 ** -24 + 1e-5) * PV)
    err = np.abs(O - Or)
    assert np.all(np.isfinite(O)) and np.all(err <= bound), float(np.max(err - bound))
    assert np.max(np.abs(to_host64(lse) - lr)) <= 1e-3
