"""The seeded input generator: determinism, rounding and recipe."""
import numpy as np

import seeded_inputs as si


def test_bf16_rounding_is_nearest_even():
    # 1 + 2^-8 lies halfway between bf16 1.0 and 1 + 2^-7: ties go to even (1.0)
    # 1 + 3*2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6: ties go to even (1 + 2^-6)
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -2.5,
                  3.0e38, 1e-40], dtype=np.float32)
    bits = si.f32_to_bf16_bits(x)
    assert bits.dtype == np.uint16
    assert list(bits[:5]) == [0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xC020]
    # large finite values stay finite; subnormals keep their top bits
    assert bits[5] == 0x7F62
    assert bits[6] == (np.array([1e-40], np.float32).view(np.uint32)[0] + 0x7FFF) >> 16


def test_f16_rounding_is_nearest_even():
    x = np.array([1 + 2 ** -11, 1 + 3 * 2 ** -11], dtype=np.float32)
    h = si.round_to_storage(x, "f16")
    assert list(h.view(np.uint16)) == [0x3C00, 0x3C02]


def test_make_qkv_is_seeded_and_ordered():
    q1, k1, v1 = si.make_qkv(1, 2, 5, 4, "f16", seed=3)
    q2, k2, v2 = si.make_qkv(1, 2, 5, 4, "f16", seed=3)
    assert q1.dtype == np.float16 and q1.shape == (1, 2, 5, 4)
    assert np.array_equal(q1, q2) and np.array_equal(k1, k2) and np.array_equal(v1, v2)
    # Q, then K, then V from one PCG64 stream
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 2, 5, 4), dtype=np.float32).astype(np.float16)
    k = rng.standard_normal((1, 2, 5, 4), dtype=np.float32).astype(np.float16)
    assert np.array_equal(q, q1) and np.array_equal(k, k1)


def test_qk_multiplier_is_exact_and_spares_v():
    q1, k1, v1 = si.make_qkv(1, 1, 16, 8, "bf16", seed=0)
    q2, k2, v2 = si.make_qkv(1, 1, 16, 8, "bf16", seed=0, qk_mult=2.0)
    # doubling adds one to the bf16 exponent field (no subnormals at N(0,1))
    assert np.array_equal(q2.astype(np.int32) - q1.astype(np.int32),
                          np.full(q1.shape, 0x80, np.int32) * (q1 & 0x7FFF != 0))
    assert np.array_equal(v1, v2)


def test_workloads():
    w = si.WORKLOADS[si.BENCH_WORKLOAD]
    assert (w.B, w.H, w.N, w.d, w.dtype) == (2, 32, 8192, 128, "bf16")
    assert set(w.causal) == {False, True}
    assert w.scale == float(np.float32(1 / np.sqrt(128)))
    long = si.WORKLOADS["mha_b1_h32_n32768_d128_bf16_causal_qk2"]
    assert long.qk_mult == 2.0 and long.causal == (True,)
