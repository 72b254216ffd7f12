"""The seeded input generator: determinism, rounding and recipe."""
import numpy as np
import pytest

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


def test_e4m3_rounding_matches_the_library():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 60,
                        rng.standard_normal(20000).astype(np.float32) * 1e-3,
                        np.array([448, -448, 0, -0.0, 2 ** -10, 3 * 2 ** -10, 1.0625, 1.1875,
                                  2 ** -6, -1.5 * 2 ** -9, 17, 464 - 1e-3], dtype=np.float32)])
    x = np.clip(x, -448, 448)
    mine = si.f32_to_e4m3_bits(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(mine, ref)
    with pytest.raises(ValueError):
        si.f32_to_e4m3_bits(np.array([500.0]))
    # a strided sweep over every fp32 bit pattern up to 448, both signs
    u = np.arange(0, 0x43E00001, 97, dtype=np.uint32)
    x = np.concatenate([u, u | np.uint32(0x80000000)]).view(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(si.f32_to_e4m3_bits(x), ref)


def test_fp8_inputs_use_the_full_range():
    q, k, v, sc = si.make_qkv_fp8(2, 3, 50, 16, seed=3)
    for t, s in zip((q, k, v), sc):
        assert t.dtype == np.uint8 and t.shape == (2, 3, 50, 16)
        assert int((t & 0x7F).max()) == 0x7E          # the largest magnitude maps to 448
        assert s > 0 and s == float(np.float32(s))
    # the same fp32 draws as the 16-bit generator, scaled
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 50, 16), dtype=np.float32)
    assert np.float32(np.max(np.abs(x)) / np.float32(448.0)) == np.float32(sc[0])


def test_dyadic_fp8_inputs_have_small_integer_scores():
    torch = pytest.importorskip("torch")
    q8, k8, v8 = si.make_qkv_fp8_dyadic(2, 3, 40, 128, seed=7)

    def dec(c):
        return torch.from_numpy(c).view(torch.float8_e4m3fn).double().numpy()

    q, k, v = dec(q8), dec(k8), dec(v8)
    assert set(np.unique(q)) <= {-1.0, 0.0, 1.0}
    assert np.all((q != 0).sum(axis=-1) == 2)
    assert set(np.unique(k)) == {-2.0, -1.0, 0.0, 1.0, 2.0}
    assert np.all(np.isfinite(v)) and len(np.unique(v8)) > 200
    s = np.einsum("bhid,bhjd->bhij", q, k)
    assert np.all(s == np.round(s)) and s.min() >= -4 and s.max() <= 4
    assert len(np.unique(s)) >= 7
    _, _, vb = si.make_qkv_fp8_dyadic(2, 3, 40, 128, seed=7, v_binade=True)
    vals = np.abs(dec(vb))
    assert vals.min() >= 1.0 and vals.max() < 2.0 and len(np.unique(vb)) == 16


# ------------------------------------------------ the paper's benchmark setting
def _golden_setting():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "benchmark_setting.txt")
    out = {}
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if line:
            key, *vals = line.split()
            out[key] = vals
    return out


def test_grid_workloads_follow_the_paper_setting():
    """The bf16 and FP8 grid workloads are the paper's stated configuration:
    every sequence length, 16k tokens per batch, hidden 2048 split into heads
    of 64 or 128, both masks (FP8: d = 128, causal)."""
    g = _golden_setting()
    seqlens = [int(x) for x in g["seqlens"]]
    tokens, hidden = int(g["tokens_per_batch"][0]), int(g["hidden"][0])
    assert list(si.GRID_N) == seqlens
    assert sorted(si.GRID_D) == sorted(int(x) for x in g["head_dims"])
    heads = {64: int(g["heads_at_head_dim_64"][0]), 128: int(g["heads_at_head_dim_128"][0])}
    masks = {"none": False, "causal": True}
    for d in si.GRID_D:
        assert heads[d] * d == hidden
        for n in seqlens:
            w = si.GRID[f"grid_d{d}_n{n}"]
            assert (w.B * w.N, w.H, w.d, w.kv_heads, w.d_v) == (tokens, heads[d], d, w.H, d)
            assert set(w.causal) == {masks[m] for m in g["masks"]}
    d8 = int(g["fp8_head_dim"][0])
    for n in seqlens:
        w = si.GRID_FP8[f"grid_fp8_d128_n{n}"]
        assert (w.dtype, w.B * w.N, w.H * w.d, w.d) == ("e4m3", tokens, hidden, d8)
        assert set(w.causal) == {masks[m] for m in g["fp8_masks"]}


def test_flop_count_is_the_paper_formula():
    """bench.py's count is the paper's 4 * seqlen^2 * head_dim * heads per
    sequence (times the batch), halved under the causal mask; the MLA shape
    counts its two products with their own head dimensions."""
    import bench
    g = _golden_setting()
    factor = int(g["flops_factor"][0])
    for w in list(si.GRID.values()):
        f = factor * w.N ** 2 * w.d * w.H * w.B
        assert bench.flops(w.B, w.H, w.N, w.d, False) == f
        assert bench.flops(w.B, w.H, w.N, w.d, True) == f / 2
    e, r = int(g["mla_embedding_dim"][0]), int(g["mla_rope_dim"][0])
    w = si.WORKLOADS["mla_b2_h128_n8192_d192_dv128_bf16_causal"]
    assert (w.d, w.d_v) == (e + r, e)
    assert bench.flops(w.B, w.H, w.N, w.d, False, w.d_v) == 2 * w.B * w.H * w.N ** 2 * (2 * e + r)


def test_grouped_workloads_use_the_paper_head_counts():
    g = _golden_setting()
    pairs = {tuple(int(x) for x in p.split("/")) for p in g["gqa_heads"]}
    found = {(w.H, w.kv_heads) for w in si.WORKLOADS.values()
             if w.kv_heads != w.H and w.N == 8192 and w.H > 32}
    assert pairs <= found


def test_periodic_inputs_repeat_the_small_draw():
    q, k, v = si.make_qkv_periodic_bnhd(2, 4, 23, 8, "bf16", period=5, seed=9, Hkv=2)
    q0, k0, v0 = si.make_qkv(2, 4, 5, 8, "bf16", seed=9, Hkv=2)
    assert q.shape == (2, 23, 4, 8) and k.shape == (2, 23, 2, 8) and q.flags.c_contiguous
    for big, small in ((q, q0), (k, k0), (v, v0)):
        for t in range(23):
            assert np.array_equal(big[:, t], small[:, :, t % 5])
