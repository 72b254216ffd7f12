"""CPU checks of the whole-output comparison used by the long GPU parity tests
(``tests/oracle_pool.py``): the oracle's own result, rounded to the output
type, passes the gate; one element moved past the gate fails it, and the
failure names that element; grouped heads and FP8 inputs take the same path.
"""
from __future__ import annotations

import numpy as np
import pytest

import seeded_inputs as si
from oracle import attention_fp64
from tests import oracle_pool
from tests.gpu_util import o_bound


def _round_bits(O: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f16":
        return O.astype(np.float16).view(np.uint16)
    return si.f32_to_bf16_bits(O.astype(np.float32))


@pytest.mark.parametrize("dtype,Hkv,causal", [("bf16", 3, False), ("f16", 3, True),
                                              ("bf16", 1, True)])
def test_rounded_oracle_passes_and_a_planted_error_fails(dtype, Hkv, causal):
    B, H, N, d = 2, 3, 97, 64
    q, k, v = si.make_qkv(B, H, N, d, dtype, seed=4, Hkv=Hkv)
    scale = si.default_scale(d)
    O, lse = attention_fp64(q, k, v, scale, causal, dtype)
    bits = _round_bits(O, dtype)
    st = oracle_pool.full_compare(q, k, v, bits, lse.astype(np.float32), scale, causal, dtype,
                                  what=f"rounded oracle {dtype}")
    assert st["bad"] == 0 and st["n"] == O.size
    assert st["max_err"] <= float(o_bound(O, dtype).max())
    # one element pushed just past the gate
    bad = O.copy()
    idx = (1, 2, 50, 7)
    bad[idx] += 1.5 * float(o_bound(O[idx], dtype))
    with pytest.raises(AssertionError, match=r"1 O elements outside the gate; worst at "
                                             r"\(1, 2, 50, 7\)"):
        oracle_pool.full_compare(q, k, v, _round_bits(bad, dtype), lse.astype(np.float32),
                                 scale, causal, dtype, what="planted")
    # an lse error above 1e-3
    lbad = lse.astype(np.float32).copy()
    lbad[0, 1, 3] += 2e-3
    with pytest.raises(AssertionError, match="lse err"):
        oracle_pool.full_compare(q, k, v, bits, lbad, scale, causal, dtype, what="planted lse")


def test_fp8_inputs_use_the_rounding_bound():
    w = si.WORKLOADS["fp8_gqa_b2_h6_kv2_n555_d128"]
    q8, k8, v8, scales = w.fp8_inputs()
    O, lse = attention_fp64(q8, k8, v8, w.scale, True, "e4m3", descale=scales)
    bits = si.f32_to_bf16_bits(O.astype(np.float32))
    st = oracle_pool.full_compare(q8, k8, v8, bits, lse.astype(np.float32), w.scale, True,
                                  "e4m3", what="rounded FP8 oracle", descale=scales)
    assert st["bad"] == 0
    bad = O.copy()
    bad[0, 5, 554, 127] += 1.0
    with pytest.raises(AssertionError, match=r"\(0, 5, 554, 127\)"):
        oracle_pool.full_compare(q8, k8, v8, si.f32_to_bf16_bits(bad.astype(np.float32)),
                                 lse.astype(np.float32), w.scale, True, "e4m3", what="planted",
                                 descale=scales)
