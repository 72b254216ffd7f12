"""Seeded synthetic attention inputs, shared by the oracle side and the HIP side.

This module draws Q, K and V and rounds them to the 16-bit storage type. It
holds none of the attention arithmetic: the oracle (``oracle/``) and the HIP
library each decode and compute on their own.

Recipe (the paper benchmarks on unstated, presumably random inputs; these
stand in for its long-context workloads of the Evaluation section's
"Benchmark setting"):

* ``rng = numpy.random.default_rng(seed)`` (PCG64), seed 0 unless stated;
* draw ``standard_normal(shape, float32)`` for Q, then K, then V; Q has shape
  ``[B, H, N, d]`` and K, V ``[B, Hkv, N, d]`` (Hkv = H unless a grouped-query
  workload names fewer key/value heads; V's last dimension is d_v when a
  workload gives values their own head dimension);
* optionally multiply Q and K by an exact power of two in fp32 (the sharper
  long-context workload uses 2);
* round to fp16 (numpy's cast, round-to-nearest-even) or to bf16 with
  round-to-nearest-even on the fp32 bit pattern.

bf16 arrays are returned as ``uint16`` bit patterns, because numpy has no
bfloat16 type; fp16 arrays are ``numpy.float16``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

DTYPES = ("f16", "bf16")   # 16-bit storage types of make_qkv; "e4m3" uses make_qkv_fp8


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even); return the uint16 bits.

    Finite inputs only (the generator never produces inf or NaN).
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    rounded = u + np.uint32(0x7FFF) + lsb
    return (rounded >> np.uint32(16)).astype(np.uint16)


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round an fp32 array to the 16-bit storage type named by ``dtype``."""
    if dtype == "f16":
        return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}; expected one of {DTYPES}")


def make_qkv(B: int, H: int, N: int, d: int, dtype: str, seed: int = 0,
             qk_mult: float = 1.0, Hkv: int | None = None, dv: int | None = None):
    """Draw Q [B, H, N, d], K [B, Hkv, N, d] and V [B, Hkv, N, dv], rounded to
    ``dtype``.

    ``Hkv`` defaults to H and ``dv`` to d.  Returns three contiguous arrays
    (``float16`` or bf16 ``uint16`` bits).
    """
    if dtype not in DTYPES:
        raise ValueError(f"unknown dtype {dtype!r}")
    Hkv = H if Hkv is None else Hkv
    dv = d if dv is None else dv
    rng = np.random.default_rng(seed)
    out = []
    for name in ("q", "k", "v"):
        shape = {"q": (B, H, N, d), "k": (B, Hkv, N, d), "v": (B, Hkv, N, dv)}[name]
        x = rng.standard_normal(shape, dtype=np.float32)
        if name in ("q", "k") and qk_mult != 1.0:
            x *= np.float32(qk_mult)
        out.append(round_to_storage(x, dtype))
        del x
    return tuple(out)


def make_qkv_periodic_bnhd(B: int, H: int, N: int, d: int, dtype: str, period: int,
                           seed: int = 0, Hkv: int | None = None):
    """Large inputs at the cost of small ones: Q, K and V are drawn as
    ``make_qkv`` draws them for ``period`` tokens and repeated along the token
    axis up to N tokens (token t holds the draw of token t mod period).  They
    are returned contiguous in [B][N][heads][d] order.  An odd period keeps
    rows whose distance is a power of two distinct, so an address that wraps
    at a power of two reads different data."""
    q0, k0, v0 = make_qkv(B, H, period, d, dtype, seed=seed, Hkv=Hkv)
    out = []
    for x in (q0, k0, v0):
        xt = np.swapaxes(x, 1, 2)                     # [B][period][heads][d]
        y = np.empty((B, N) + xt.shape[2:], dtype=x.dtype)
        for t in range(0, N, period):
            n = min(period, N - t)
            y[:, t:t + n] = xt[:, :n]
        out.append(y)
    return tuple(out)


# ---------------------------------------------------------------- FP8 inputs
# OCP E4M3FN: 1 sign, 4 exponent (bias 7) and 3 mantissa bits; no infinities;
# S.1111.111 is NaN; the largest finite value is 448.
E4M3_MAX = 448.0


def f32_to_e4m3_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values with |x| <= 448 to OCP E4M3FN, to nearest with
    ties to the even code (the even mantissa); return the uint8 codes.

    Normal results (|x| >= 2^-6): round the fp32 significand to 3 bits on the
    bit pattern; the code is then (exponent + 7) << 3 | mantissa.  Subnormal
    results: the code is |x| / 2^-9 rounded half to even (8 there is 2^-6,
    which is code 8 as well)."""
    x = np.asarray(x)
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if x.dtype != np.float32 and not np.array_equal(x32, x):
        raise ValueError("inputs must be fp32 values")
    a = np.abs(x32)
    if not np.all(a <= np.float32(E4M3_MAX)):
        raise ValueError("values beyond the E4M3 range (448) or NaN")
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(20)) & np.uint32(1)
    r = (u + np.uint32(0x7FFFF) + lsb) >> np.uint32(20)          # sign 0, 8-bit exponent, 3 bits
    normal = (((r >> np.uint32(3)).astype(np.int32) - 127 + 7) << 3) | (r & np.uint32(7)).astype(np.int32)
    sub = np.rint(a * np.float32(512.0)).astype(np.int32)
    code = np.where(a >= np.float32(2.0 ** -6), normal, sub).astype(np.uint8)
    return np.where(np.signbit(x32), code | np.uint8(0x80), code).astype(np.uint8)   # keeps -0


def make_qkv_fp8(B: int, H: int, N: int, d: int, seed: int = 0, Hkv: int | None = None):
    """FP8 inputs: Q, K, V drawn as ``make_qkv`` draws them (fp32 normals, Q then
    K then V; K and V with ``Hkv`` heads, default H), each scaled per tensor so
    that its largest magnitude maps to 448, rounded to E4M3.  Returns (q8, k8,
    v8, scales) with uint8 codes and the three float32 descale factors: the
    real tensor is scale * decode(code)."""
    Hkv = H if Hkv is None else Hkv
    rng = np.random.default_rng(seed)
    out, scales = [], []
    for heads in (H, Hkv, Hkv):
        x = rng.standard_normal((B, heads, N, d), dtype=np.float32)
        s = np.float32(np.max(np.abs(x)) / np.float32(E4M3_MAX))
        y = np.minimum(np.abs(x / s), np.float32(E4M3_MAX)) * np.sign(x)
        out.append(f32_to_e4m3_bits(y))
        scales.append(float(s))
        del x, y
    return out[0], out[1], out[2], tuple(scales)


def make_qkv_fp8_dyadic(B: int, H: int, N: int, d: int, seed: int = 0,
                        v_binade: bool = False, Hkv: int | None = None):
    """FP8 inputs with small integer dot products.  Each Q row holds +1 or -1
    (even odds) at two distinct columns drawn uniformly and zeros elsewhere; K
    entries are integers drawn uniformly from -2 .. 2; V holds codes drawn
    uniformly from the 254 finite E4M3 codes (every exponent, subnormals and
    both zeros included), or with ``v_binade`` from the 16 codes of [1, 2)
    and (-2, -1] (random sign and mantissa).  Every q . k is then an integer
    in [-4, 4].  K and V have ``Hkv`` heads (default H).  Returns uint8 codes
    (q8, k8, v8); the caller picks the scale factors."""
    Hkv = H if Hkv is None else Hkv
    rng = np.random.default_rng(seed)
    cols = np.argsort(rng.random((B, H, N, d)), axis=-1)[..., :2]
    signs = rng.choice(np.array([-1.0, 1.0], dtype=np.float32), size=(B, H, N, 2))
    q = np.zeros((B, H, N, d), dtype=np.float32)
    np.put_along_axis(q, cols, signs, axis=-1)
    k = rng.integers(-2, 3, size=(B, Hkv, N, d)).astype(np.float32)
    if v_binade:
        pool = np.array([s << 7 | 7 << 3 | m for s in (0, 1) for m in range(8)], dtype=np.uint8)
    else:
        pool = np.array([c for c in range(256) if c & 0x7F != 0x7F], dtype=np.uint8)
    v = pool[rng.integers(0, pool.size, size=(B, Hkv, N, d))]
    return f32_to_e4m3_bits(q), f32_to_e4m3_bits(k), v


def default_scale(d: int) -> float:
    """The softmax scale 1/sqrt(d), as the fp32 value handed to the kernel."""
    return float(np.float32(1.0 / np.sqrt(np.float64(d))))


@dataclass(frozen=True)
class Workload:
    """One synthetic attention workload: shapes, storage type, masks, input recipe."""
    name: str
    B: int
    H: int
    N: int
    d: int
    dtype: str
    causal: tuple = field(default=(False,))
    qk_mult: float = 1.0
    seed: int = 0
    Hkv: int = 0          # key/value heads; 0 means H (multi-head attention)
    dv: int = 0           # head dimension of V and O; 0 means d

    @property
    def kv_heads(self) -> int:
        return self.Hkv or self.H

    @property
    def d_v(self) -> int:
        return self.dv or self.d

    @property
    def scale(self) -> float:
        return default_scale(self.d)   # 1/sqrt of the query/key head dimension

    def inputs(self):
        if self.dtype == "e4m3":
            raise ValueError("FP8 workloads draw their inputs with fp8_inputs()")
        return make_qkv(self.B, self.H, self.N, self.d, self.dtype,
                        seed=self.seed, qk_mult=self.qk_mult, Hkv=self.kv_heads, dv=self.d_v)

    def fp8_inputs(self):
        """(q8, k8, v8, (q_scale, k_scale, v_scale)) of an FP8 workload."""
        return make_qkv_fp8(self.B, self.H, self.N, self.d, seed=self.seed, Hkv=self.kv_heads)


WORKLOADS = {
    w.name: w for w in (
        Workload("mha_b1_h2_n128_d64_f16", 1, 2, 128, 64, "f16", (False,)),
        Workload("mha_b8_h16_n1024_d64_f16", 8, 16, 1024, 64, "f16", (False,)),
        Workload("mha_b4_h32_n2048_d128_f16_causal", 4, 32, 2048, 128, "f16", (True,)),
        Workload("mha_b2_h32_n8192_d128_bf16", 2, 32, 8192, 128, "bf16", (False, True)),
        Workload("mha_b1_h32_n32768_d128_bf16_causal_qk2", 1, 32, 32768, 128, "bf16",
                 (True,), qk_mult=2.0),
        # grouped-query and multi-query attention: the appendix table's LLM head
        # configurations (64 query / 8 key-value heads, 128 / 8; d = 128, causal)
        # at the 16k-token budget of the benchmark grid, plus MQA and small cases
        Workload("gqa_b2_h64_kv8_n8192_d128_bf16_causal", 2, 64, 8192, 128, "bf16", (True,),
                 Hkv=8),
        Workload("gqa_b2_h128_kv8_n8192_d128_bf16_causal", 2, 128, 8192, 128, "bf16", (True,),
                 Hkv=8),
        Workload("mqa_b2_h32_kv1_n8192_d128_bf16", 2, 32, 8192, 128, "bf16", (False, True),
                 Hkv=1),
        Workload("gqa_b2_h8_kv2_n1000_d64_f16", 2, 8, 1000, 64, "f16", (False, True), Hkv=2),
        Workload("mqa_b2_h6_kv1_n777_d128_bf16", 2, 6, 777, 128, "bf16", (False, True), Hkv=1),
        # the MLA shape in explicit form: head dimension 128 plus a 64-wide RoPE
        # part for queries and keys (d = 192), values and outputs 128 wide, with
        # DeepSeek-V3's 128 heads at the 16k-token budget, causal (the paper's
        # MLA table), plus smaller cases
        Workload("mla_b2_h128_n8192_d192_dv128_bf16_causal", 2, 128, 8192, 192, "bf16",
                 (True,), dv=128),
        Workload("mla_b1_h16_n4096_d192_dv128_bf16", 1, 16, 4096, 192, "bf16",
                 (False, True), dv=128),
        Workload("mla_b2_h4_n777_d192_dv128_f16", 2, 4, 777, 192, "f16", (False, True), dv=128),
        # FP8 (OCP E4M3) inputs with per-tensor scales, bf16 output: the paper's
        # FP8 table is MHA with the causal mask at d = 128
        Workload("fp8_b2_h32_n8192_d128", 2, 32, 8192, 128, "e4m3", (False, True)),
        Workload("fp8_b2_h3_n333_d128", 2, 3, 333, 128, "e4m3", (False, True)),
        # FP8 with the appendix's grouped-query heads (64 query / 8 key-value)
        Workload("fp8_gqa_b2_h64_kv8_n8192_d128_causal", 2, 64, 8192, 128, "e4m3", (True,),
                 Hkv=8),
        Workload("fp8_gqa_b2_h6_kv2_n555_d128", 2, 6, 555, 128, "e4m3", (False, True), Hkv=2),
    )
}

# The paper's benchmark grid (Evaluation, "Benchmark setting"): sequence length
# 512 .. 16k at a fixed 16k tokens per batch (B = 16384 / N), hidden size 2048
# (H = 2048 / d), head dimension 64 or 128, with and without the causal mask.
GRID_N = (512, 1024, 2048, 4096, 8192, 16384)
GRID_D = (64, 128)
GRID = {
    f"grid_d{d}_n{n}": Workload(f"grid_d{d}_n{n}", 16384 // n, 2048 // d, n, d, "bf16",
                                (False, True))
    for d in GRID_D for n in GRID_N
}
WORKLOADS.update(GRID)
# The paper's FP8 table: the same grid at d = 128, causal mask only.
GRID_FP8 = {
    f"grid_fp8_d128_n{n}": Workload(f"grid_fp8_d128_n{n}", 16384 // n, 2048 // 128, n, 128,
                                    "e4m3", (True,))
    for n in GRID_N
}
WORKLOADS.update(GRID_FP8)

# The workload the throughput figure is quoted on (N = 8192, d = 128).
BENCH_WORKLOAD = "mha_b2_h32_n8192_d128_bf16"
# The small workload that the full oracle finishes in well under a second.
SMOKE_WORKLOAD = "mha_b1_h2_n128_d64_f16"
