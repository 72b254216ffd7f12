"""The checking build (``libqm_attn_debug.so``: the same sources compiled with
-DQM_DEBUG_SYNC, a barrier after every key block on top of the K/V ring
protocol's own) must give byte-identical outputs to the release build.

The release kernels publish a pair of 64-key blocks per barrier through
four-slot LDS rings (two-slot rings, one barrier per block, for 192-wide
keys and four-wave workgroups), and the FP8 and d = 64 instances run a
block's second product one block later from a V slot the ring keeps alive.
Extra barriers only remove overlap between waves; if the release protocol
let a wave read a slot before its loads had landed, or load into a slot
another wave still read, the two builds would disagree.  Covered: the bench
workload (both masks), FP8, d = 64 in both workgroup sizes, ragged lengths,
grouped heads, the MLA shape and [B][N][H][d].
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import seeded_inputs as si
from tests.gpu_util import to_device

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def libs():
    import torch
    import paper_2506_12355_amd as qa
    assert torch.cuda.is_available()
    return qa.load_library(), qa.open_library(qa.DEBUG_LIB_PATH)


def _run(lib, tq, tk, tv, o, lse, B, H, Hkv, N, d, dv, scale, causal, dtype, layout=0,
         fp8_scales=None):
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    o.fill_(float("nan"))
    lse.fill_(float("nan"))
    ptrs = (tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), o.data_ptr(), lse.data_ptr())
    if fp8_scales is not None:
        st = lib.qm_attn_fwd_fp8_layout(*ptrs, B, H, Hkv, N, d, *fp8_scales, scale, int(causal),
                                        stream, layout)
    else:
        st = lib.qm_attn_fwd_layout(*ptrs, B, H, Hkv, N, d, dv, scale, int(causal), stream,
                                    dtype, layout)
    assert st == 0, st
    torch.cuda.synchronize()
    return o.view(torch.int16).clone(), lse.view(torch.int32).clone()


def _both(libs, what, tq, tk, tv, B, H, Hkv, N, d, dv, scale, dtype, layout=0, fp8_scales=None,
          tiles=(0,)):
    import torch
    odt = torch.bfloat16 if fp8_scales is not None or dtype == 1 else torch.float16
    oshape = (B, N, H, dv) if layout else (B, H, N, dv)
    o = torch.empty(oshape, dtype=odt, device="cuda")
    lse = torch.empty((B, H, N), dtype=torch.float32, device="cuda")
    for rows in tiles:
        for lib in libs:
            assert lib.qm_attn_set_tile_rows(rows) == 0
        for causal in (False, True):
            _say(f"case {what} tile_rows={rows or 'auto'} causal={causal}")
            rel = _run(libs[0], tq, tk, tv, o, lse, B, H, Hkv, N, d, dv, scale, causal, dtype,
                       layout, fp8_scales)
            dbg = _run(libs[1], tq, tk, tv, o, lse, B, H, Hkv, N, d, dv, scale, causal, dtype,
                       layout, fp8_scales)
            assert torch.equal(rel[0], dbg[0]), f"{what}: O differs from the checking build"
            assert torch.equal(rel[1], dbg[1]), f"{what}: lse differs from the checking build"
    for lib in libs:
        lib.qm_attn_set_tile_rows(0)


@pytest.mark.parametrize("name", ["mha_b2_h32_n8192_d128_bf16", "grid_d64_n8192",
                                  "mha_b8_h16_n1024_d64_f16", "mha_b4_h32_n2048_d128_f16_causal",
                                  "gqa_b2_h64_kv8_n8192_d128_bf16_causal",
                                  "mla_b1_h16_n4096_d192_dv128_bf16"])
def test_16bit_workloads_match_checking_build(libs, name):
    w = si.WORKLOADS[name]
    q, k, v = w.inputs()
    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    dtype = 1 if w.dtype == "bf16" else 0
    tiles = (128, 256) if w.d != 192 and w.N <= 2048 else (0,)
    _both(libs, name, tq, tk, tv, w.B, w.H, w.kv_heads, w.N, w.d, w.d_v, w.scale, dtype,
          tiles=tiles)


@pytest.mark.parametrize("N,d,dtype", [(1000, 64, "f16"), (1000, 128, "bf16"), (4161, 64, "bf16"),
                                       (3001, 128, "f16"), (65, 128, "bf16")])
def test_ragged_lengths_match_checking_build(libs, N, d, dtype):
    q, k, v = si.make_qkv(2, 3, N, d, dtype, seed=N + d)
    tq, tk, tv = (to_device(x, dtype) for x in (q, k, v))
    _both(libs, f"N={N} d={d} {dtype}", tq, tk, tv, 2, 3, 3, N, d, d, si.default_scale(d),
          1 if dtype == "bf16" else 0, tiles=(128, 256))


def test_bnhd_layout_matches_checking_build(libs):
    q, k, v = si.make_qkv(2, 8, 3000, 128, "bf16", seed=77, Hkv=2)
    tq, tk, tv = (to_device(np.ascontiguousarray(np.swapaxes(x, 1, 2)), "bf16")
                  for x in (q, k, v))
    _both(libs, "[B][N][H][d] 8/2 heads", tq, tk, tv, 2, 8, 2, 3000, 128, 128,
          si.default_scale(128), 1, layout=1)


@pytest.mark.parametrize("name", ["fp8_b2_h32_n8192_d128", "fp8_gqa_b2_h6_kv2_n555_d128",
                                  "grid_fp8_d128_n2048"])
def test_fp8_workloads_match_checking_build(libs, name):
    import torch
    w = si.WORKLOADS[name]
    q8, k8, v8, scales = w.fp8_inputs()
    tq, tk, tv = (torch.from_numpy(x).cuda() for x in (q8, k8, v8))
    _both(libs, name, tq, tk, tv, w.B, w.H, w.kv_heads, w.N, w.d, w.d, w.scale, 2,
          fp8_scales=scales, tiles=(128, 256))
