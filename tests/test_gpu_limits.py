"""GPU parity at the size limits the front end accepts.

* ``[B][N][H][d]`` at the largest N whose padded rows still fit the kernels'
  32-bit byte offsets: (N + 256) * H * d * 2 = 2^32 - 2^14 with H = 64,
  d = 128 (four 4 GiB tensors).  Inputs repeat with an odd period, so a row
  address that wrapped at any power of two would read different data.
* One head of 2^20 + 17 tokens in ``[B][H][N][d]`` (d = 64, f16).
* Many small heads (3003 workgroups, not a multiple of the eight XCDs), and
  multi-query attention with 4096 query heads on one key/value head.

Rows are sampled where the long sequences end and around the 2^31-byte mark;
the small shapes are compared in full.
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


def test_bnhd_at_the_32_bit_offset_limit(qa):
    import torch
    B, H, d = 1, 64, 128
    N = (1 << 18) - 257                       # (N + 256) * H * d * 2 = 2^32 - 2^14
    assert (N + 256) * H * d * 2 < 1 << 32 <= (N + 257) * H * d * 2
    _say(f"case BNHD limit: drawing B={B} N={N} H={H} d={d} bf16 (period 3001)")
    q, k, v = si.make_qkv_periodic_bnhd(B, H, N, d, "bf16", period=3001, seed=101)
    tq, tk, tv = (to_device(x, "bf16") for x in (q, k, v))
    scale = si.default_scale(d)
    # [B][H][N][d] views of the same host arrays for the oracle
    qh, kh, vh = (np.swapaxes(x, 1, 2) for x in (q, k, v))
    rng = np.random.default_rng(102)
    rows = ([(0, 0, N - 1), (0, H - 1, N - 1), (0, 31, N - 2), (0, 7, N - 257),
             (0, 17, 131071), (0, 17, 131072), (0, 40, (1 << 17) + 3001), (0, 5, 0)]
            + [(0, int(rng.integers(H)), int(rng.integers(N))) for _ in range(6)])
    for causal in (False, True):
        _say(f"case BNHD limit causal={causal}: running")
        o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=scale, layout="bnhd")
        torch.cuda.synchronize()
        assert bool(torch.isfinite(lse).all())
        O = np.array([to_host64(o[b, i, h]) for b, h, i in rows])
        L = np.array([float(lse[b, h, i]) for b, h, i in rows])
        _say(f"case BNHD limit causal={causal}: oracle on {len(rows)} rows")
        Or, lr = attention_rows_fp64(qh, kh, vh, scale, causal, "bf16", rows)
        check_close(O, L, Or, lr, "bf16", f"BNHD limit N={N} causal={causal}")
        del o, lse
        torch.cuda.empty_cache()


def test_one_head_of_a_million_tokens(qa):
    import torch
    B, H, N, d = 1, 2, (1 << 20) + 17, 64
    _say(f"case long head: drawing B={B} H={H} N={N} d={d} f16")
    q, k, v = si.make_qkv(B, H, N, d, "f16", seed=103)
    tq, tk, tv = (to_device(x, "f16") for x in (q, k, v))
    scale = si.default_scale(d)
    rows = [(0, 0, 0), (0, 1, 1), (0, 0, N - 1), (0, 1, N - 1), (0, 1, N - 18),
            (0, 0, 1 << 19), (0, 1, (1 << 20) - 1), (0, 0, 1 << 20), (0, 1, 777777)]
    for causal in (False, True):
        _say(f"case long head causal={causal}: running")
        o, lse = qa.fwd(tq, tk, tv, causal=causal, scale=scale)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
        O = np.array([to_host64(o[b, h, i]) for b, h, i in rows])
        L = np.array([float(lse[b, h, i]) for b, h, i in rows])
        Or, lr = attention_rows_fp64(q, k, v, scale, causal, "f16", rows)
        check_close(O, L, Or, lr, "f16", f"long head N={N} causal={causal}")


def test_many_small_heads(qa):
    """3 x 1001 heads of 33 tokens: 3003 one-block workgroups, a count that
    leaves a tail after the per-XCD remapping."""
    import torch
    B, H, N, d = 3, 1001, 33, 64
    q, k, v = si.make_qkv(B, H, N, d, "f16", seed=104)
    scale = si.default_scale(d)
    for causal in (False, True):
        _say(f"case many heads causal={causal}")
        o, lse = qa.fwd(*(to_device(x, "f16") for x in (q, k, v)), causal=causal, scale=scale)
        torch.cuda.synchronize()
        Or, lr = attention_fp64(q, k, v, scale, causal, "f16")
        check_close(to_host64(o), to_host64(lse), Or, lr, "f16",
                    f"many heads causal={causal}")


def test_multi_query_with_4096_query_heads(qa):
    import torch
    B, H, Hkv, N, d = 1, 4096, 1, 65, 128
    q, k, v = si.make_qkv(B, H, N, d, "bf16", seed=105, Hkv=Hkv)
    scale = si.default_scale(d)
    for causal in (False, True):
        _say(f"case MQA 4096/1 causal={causal}")
        o, lse = qa.fwd(*(to_device(x, "bf16") for x in (q, k, v)), causal=causal,
                        scale=scale)
        torch.cuda.synchronize()
        Or, lr = attention_fp64(q, k, v, scale, causal, "bf16")
        check_close(to_host64(o), to_host64(lse), Or, lr, "bf16",
                    f"MQA 4096/1 causal={causal}")
