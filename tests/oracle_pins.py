"""Pins for the fp64 oracle: checks fixed by the mathematics, not by the oracle.

Each ``pin_*`` takes the oracle module (``oracle.softmax_attention``) and raises
``AssertionError`` when the module disagrees with what the definition of
attention (the paper's Background, subsection "Attention Operators and
acceleration") fixes independently of any implementation:

* a brute force in 50-digit decimal arithmetic on tiny inputs, with its own
  input decoding, no max subtraction and the explicit softmax matrix;
* closed forms (all-equal scores give the mean of the visible values);
* invariants (softmax rows sum to 1, shift invariance in K, linearity in V,
  key-permutation invariance, constant value rows);
* special cases (one key, causal row 0, causal last row, causal prefix, a
  sharp one-hot row, large scales without overflow);
* grouped-query attention: each query head against the brute force with its
  group's key/value head, equality with explicitly repeated key/value heads,
  identical query heads under multi-query attention;
* values narrower than queries and keys (the MLA shape): the brute force, and
  output columns that depend only on their own value column;
* FP8 inputs: E4M3 decoding on known codes and against the library's own
  float8 conversion, and the brute force on scaled FP8 inputs.

``tests/test_oracle.py`` runs every pin on the oracle and shows that planted
mistakes in the oracle fail at least one pin.
"""
from __future__ import annotations

import math
import struct
from decimal import Decimal, localcontext

import numpy as np

from seeded_inputs import make_qkv


# --------------------------------------------------------------------------
# independent helpers (no oracle code)
# --------------------------------------------------------------------------
def _decode_independent(x, dtype):
    """Decode stored values to Python floats without the oracle's decoder."""
    flat = np.asarray(x).reshape(-1)
    if dtype == "f16":
        out = [struct.unpack("<e", struct.pack("<H", int(u)))[0]
               for u in flat.view(np.uint16)]
    elif dtype == "bf16":
        out = [struct.unpack("<f", struct.pack("<I", int(u) << 16))[0] for u in flat]
    elif dtype == "e4m3":
        import torch   # the library's own FP8 decoding, independent of the oracle's table
        return torch.from_numpy(np.ascontiguousarray(x)).view(torch.float8_e4m3fn).double().numpy()
    elif dtype == "f64":
        out = [float(t) for t in flat]
    else:
        raise ValueError(dtype)
    return np.array(out, dtype=np.float64).reshape(np.asarray(x).shape)


def brute_force_decimal(q, k, v, scale, causal):
    """Attention for one head in 50-digit decimal arithmetic.

    q, k, v: [N, d] Python-float arrays.  No max subtraction: the decimal
    exponent range holds exp(s) for any score these tests use.  Returns
    (O [N, d], lse [N]) as floats.
    """
    N, d = q.shape
    with localcontext() as ctx:
        ctx.prec = 50
        Q = [[Decimal(float(t)) for t in row] for row in q]
        K = [[Decimal(float(t)) for t in row] for row in k]
        V = [[Decimal(float(t)) for t in row] for row in v]
        sc = Decimal(float(scale))
        O = np.empty((N, v.shape[1]))
        lse = np.empty(N)
        for i in range(N):
            keys = range(i + 1) if causal else range(N)
            e = []
            for j in keys:
                dot = sum((Q[i][c] * K[j][c] for c in range(d)), Decimal(0))
                e.append((sc * dot).exp())
            Z = sum(e, Decimal(0))
            for c in range(v.shape[1]):
                num = sum((e[t] * V[j][c] for t, j in enumerate(keys)), Decimal(0))
                O[i, c] = float(num / Z)
            lse[i] = float(Z.ln())
    return O, lse


def _close(a, b, atol, what):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.shape != b.shape:
        raise AssertionError(f"{what}: shape {a.shape} != {b.shape}")
    if not np.all(np.isfinite(a)):
        raise AssertionError(f"{what}: non-finite values")
    err = np.max(np.abs(a - b)) if a.size else 0.0
    if not err <= atol:
        raise AssertionError(f"{what}: max abs err {err:.3e} > {atol:.3e}")


# --------------------------------------------------------------------------
# pins
# --------------------------------------------------------------------------
BRUTE_CASES = [
    # (N, d, dtype, scale, causal, seed)
    (1, 1, "f16", 1.0, False, 1),
    (2, 4, "f16", 0.5, True, 2),
    (3, 4, "bf16", -0.7, False, 3),
    (5, 16, "f16", 0.25, True, 4),
    (8, 16, "bf16", 0.25, False, 5),
    (8, 4, "bf16", 0.0, True, 6),
    (7, 16, "f16", 1.0 / math.sqrt(16), True, 7),
    (6, 4, "f16", 37.5, False, 8),      # sharp softmax, scores in the hundreds
    (6, 16, "bf16", 1000.0, True, 9),   # scores ~1e4: needs the max subtraction
]


def pin_brute_force(mod):
    """Every output of the oracle equals the 50-digit brute force."""
    for N, d, dtype, scale, causal, seed in BRUTE_CASES:
        q, k, v = make_qkv(1, 2, N, d, dtype, seed=seed)
        O, lse = mod.attention_fp64(q, k, v, scale, causal, dtype, row_block=3)
        s32 = float(np.float32(scale))
        for h in range(2):
            qf = _decode_independent(q[0, h], dtype)
            kf = _decode_independent(k[0, h], dtype)
            vf = _decode_independent(v[0, h], dtype)
            Ob, lb = brute_force_decimal(qf, kf, vf, s32, causal)
            smax = abs(s32) * float(np.max(np.abs(qf @ kf.T))) + 1.0
            tol = 1e-13 + 8e-16 * d * smax
            _close(O[0, h], Ob, tol * max(1.0, float(np.max(np.abs(vf)))),
                   f"O brute N={N} d={d} {dtype} scale={scale} causal={causal}")
            _close(lse[0, h], lb, tol * max(1.0, float(np.max(np.abs(lb)))),
                   f"lse brute N={N} d={d} {dtype} scale={scale} causal={causal}")


def pin_zero_query_mean(mod):
    """Q = 0 makes every visible score equal: O_i = mean of visible V, lse = ln(count)."""
    for causal in (False, True):
        for dtype in ("f16", "bf16"):
            _, k, v = make_qkv(2, 3, 29, 8, dtype, seed=11)
            q = np.zeros_like(k)
            O, lse = mod.attention_fp64(q, k, v, 0.3, causal, dtype, row_block=8)
            vf = _decode_independent(v, dtype)
            for b in range(2):
                for h in range(3):
                    for i in range(29):
                        n = i + 1 if causal else 29
                        mean = [math.fsum(vf[b, h, :n, c]) / n for c in range(8)]
                        _close(O[b, h, i], mean, 1e-14, f"zero-Q mean causal={causal}")
                        _close(lse[b, h, i], math.log(n), 1e-14, "zero-Q lse")


def pin_zero_scale_mean(mod):
    """scale = 0 with random Q: the same closed form as Q = 0."""
    for causal in (False, True):
        q, k, v = make_qkv(1, 2, 17, 4, "f16", seed=12)
        O, lse = mod.attention_fp64(q, k, v, 0.0, causal, "f16", row_block=5)
        vf = _decode_independent(v, "f16")
        for h in range(2):
            for i in range(17):
                n = i + 1 if causal else 17
                mean = vf[0, h, :n].sum(axis=0) / n
                _close(O[0, h, i], mean, 1e-14, "zero-scale mean")
                _close(lse[0, h, i], math.log(n), 1e-14, "zero-scale lse")


def pin_softmax_rows(mod):
    """P rows sum to 1, masked entries are exactly 0, P_ij = exp(s_ij - lse_i)."""
    rng = np.random.default_rng(13)
    Q = rng.standard_normal((23, 6))
    K = rng.standard_normal((23, 6))
    for causal in (False, True):
        S = mod.scores_fp64(Q, K, 0.9, causal, row0=0)
        ref = (Q @ K.T) * 0.9
        for i in range(23):
            for j in range(23):
                if causal and j > i:
                    if not S[i, j] == -np.inf:
                        raise AssertionError("masked score is not -inf")
                elif abs(S[i, j] - ref[i, j]) > 1e-14 * max(1.0, abs(ref[i, j])):
                    raise AssertionError("visible score differs from scale*q.k")
        P, lse = mod.softmax_rows_fp64(S)
        _close(P.sum(axis=1), np.ones(23), 1e-14, "P row sums")
        for i in range(23):
            for j in range(23):
                if causal and j > i:
                    if P[i, j] != 0.0:
                        raise AssertionError("masked probability is not 0")
                elif abs(P[i, j] - math.exp(S[i, j] - lse[i])) > 1e-14:
                    raise AssertionError("P_ij != exp(s_ij - lse_i)")


def pin_shift_invariance(mod):
    """k_j -> k_j + u leaves O unchanged and shifts lse_i by scale * q_i.u."""
    rng = np.random.default_rng(14)
    q = rng.standard_normal((1, 2, 19, 5))
    k = rng.standard_normal((1, 2, 19, 5))
    v = rng.standard_normal((1, 2, 19, 5))
    u = rng.standard_normal(5)
    for causal in (False, True):
        O1, l1 = mod.attention_fp64(q, k, v, 0.8, causal, "f64", row_block=4)
        O2, l2 = mod.attention_fp64(q, k + u, v, 0.8, causal, "f64", row_block=4)
        _close(O2, O1, 1e-13, "shift-invariant O")
        _close(l2, l1 + 0.8 * (q @ u), 1e-13, "shifted lse")


def pin_constant_value_rows(mod):
    """v_j = c for every key j gives O_i = c."""
    q, k, _ = make_qkv(1, 2, 21, 8, "bf16", seed=15)
    c = np.array([1.5, -2.0, 0.25, 3.0, -0.5, 8.0, 0.0, 1.0])
    v = np.broadcast_to(c, (1, 2, 21, 8)).copy()
    qf = _decode_independent(q, "bf16")
    kf = _decode_independent(k, "bf16")
    for causal in (False, True):
        O, _ = mod.attention_fp64(qf, kf, v, 0.35, causal, "f64", row_block=6)
        _close(O, np.broadcast_to(c, O.shape), 1e-14 * 8, "constant V rows")


def pin_linear_in_v(mod):
    """O is linear in V: O(V1 + 2 V2) = O(V1) + 2 O(V2)."""
    rng = np.random.default_rng(16)
    q = rng.standard_normal((1, 1, 17, 4))
    k = rng.standard_normal((1, 1, 17, 4))
    v1 = rng.standard_normal((1, 1, 17, 4))
    v2 = rng.standard_normal((1, 1, 17, 4))
    for causal in (False, True):
        a, _ = mod.attention_fp64(q, k, v1 + 2 * v2, 0.6, causal, "f64")
        b, _ = mod.attention_fp64(q, k, v1, 0.6, causal, "f64")
        c, _ = mod.attention_fp64(q, k, v2, 0.6, causal, "f64")
        _close(a, b + 2 * c, 1e-13, "linearity in V")


def pin_key_permutation(mod):
    """Without a mask, permuting keys together with their values leaves O and lse."""
    rng = np.random.default_rng(17)
    q = rng.standard_normal((1, 1, 24, 6))
    k = rng.standard_normal((1, 1, 24, 6))
    v = rng.standard_normal((1, 1, 24, 6))
    perm = rng.permutation(24)
    O1, l1 = mod.attention_fp64(q, k, v, 0.7, False, "f64", row_block=5)
    O2, l2 = mod.attention_fp64(q, k[:, :, perm], v[:, :, perm], 0.7, False, "f64",
                                row_block=5)
    _close(O2, O1, 1e-13, "key permutation O")
    _close(l2, l1, 1e-13, "key permutation lse")


def pin_single_key(mod):
    """N = 1: O = V and lse = scale * q.k."""
    q, k, v = make_qkv(2, 2, 1, 16, "f16", seed=18)
    qf, kf, vf = (_decode_independent(t, "f16") for t in (q, k, v))
    for causal in (False, True):
        O, lse = mod.attention_fp64(q, k, v, 0.25, causal, "f16")
        _close(O, vf, 0.0, "N=1 O")
        expect = 0.25 * np.einsum("bhnd,bhnd->bhn", qf, kf)
        _close(lse, expect, 1e-14, "N=1 lse")


def pin_causal_special_rows(mod):
    """Causal row 0 is V row 0; the last causal row equals the last unmasked row;
    causal row i equals unmasked attention over keys 0..i."""
    q, k, v = make_qkv(1, 2, 33, 8, "f16", seed=19)
    vf = _decode_independent(v, "f16")
    Oc, lc = mod.attention_fp64(q, k, v, 0.4, True, "f16", row_block=7)
    On, ln = mod.attention_fp64(q, k, v, 0.4, False, "f16", row_block=7)
    _close(Oc[:, :, 0], vf[:, :, 0], 0.0, "causal row 0")
    _close(Oc[:, :, -1], On[:, :, -1], 1e-14, "causal last row")
    _close(lc[:, :, -1], ln[:, :, -1], 1e-14, "causal last lse")
    for i in (1, 5, 16, 32):
        Op, lp = mod.attention_fp64(q[:, :, :i + 1].copy(), k[:, :, :i + 1].copy(),
                                    v[:, :, :i + 1].copy(), 0.4, False, "f16")
        _close(Oc[:, :, i], Op[:, :, i], 1e-14, f"causal row {i} vs prefix")
        _close(lc[:, :, i], lp[:, :, i], 1e-14, f"causal lse {i} vs prefix")


def pin_one_hot(mod):
    """Orthogonal keys and a query aligned with key 3 at a large scale give O = V[3]."""
    N, d = 8, 8
    k = np.eye(N, d)[None, None] * 4.0
    q = np.zeros((1, 1, N, d))
    q[..., 3] = 4.0
    v = np.random.default_rng(20).standard_normal((1, 1, N, d))
    O, lse = mod.attention_fp64(q, k, v, 50.0, False, "f64")
    # every other score is 0 while key 3 scores 800: their weight is exp(-800) ~ 0
    _close(O[0, 0], np.broadcast_to(v[0, 0, 3], (N, d)), 1e-300, "one-hot row")
    _close(lse[0, 0], np.full(N, 800.0), 1e-12, "one-hot lse")


def pin_rows_match_full(mod):
    """The per-row entry point returns the same rows as the full computation."""
    for causal in (False, True):
        q, k, v = make_qkv(2, 3, 40, 8, "bf16", seed=21)
        O, lse = mod.attention_fp64(q, k, v, 0.35, causal, "bf16", row_block=16)
        rows = [(0, 0, 0), (1, 2, 39), (0, 1, 17), (1, 0, 5)]
        Or, lr = mod.attention_rows_fp64(q, k, v, 0.35, causal, "bf16", rows)
        for t, (b, h, i) in enumerate(rows):
            _close(Or[t], O[b, h, i], 1e-14, "row entry O")
            _close(lr[t], lse[b, h, i], 1e-14, "row entry lse")


def pin_decode(mod):
    """Decoding of 16-bit storage is exact on known bit patterns."""
    bf = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x3EAB, 0x8000], dtype=np.uint16)
    expect = [1.0, -2.0, 2.0 ** -133, 3.3895313892515355e38, 0.333984375, -0.0]
    got = mod.decode_fp64(bf, "bf16")
    if not list(got) == expect:
        raise AssertionError(f"bf16 decode {list(got)} != {expect}")
    hf = np.array([0x3C00, 0xC000, 0x0001, 0x7BFF, 0x3555], dtype=np.uint16).view(np.float16)
    expect = [1.0, -2.0, 2.0 ** -24, 65504.0, 0.333251953125]
    got = mod.decode_fp64(hf, "f16")
    if not list(got) == expect:
        raise AssertionError(f"f16 decode {list(got)} != {expect}")


GQA_BRUTE_CASES = [
    # (H, Hkv, N, d, dtype, scale, causal, seed)
    (4, 2, 5, 8, "f16", 0.4, True, 31),
    (3, 1, 6, 4, "bf16", 0.9, False, 32),
    (6, 3, 4, 16, "bf16", 0.25, True, 33),
    (4, 4, 3, 4, "f16", -0.5, False, 34),
]


def pin_gqa_brute_force(mod):
    """Grouped-query attention: every query head equals the 50-digit brute force
    with the key/value head of its contiguous group, index h * Hkv // H."""
    for H, Hkv, N, d, dtype, scale, causal, seed in GQA_BRUTE_CASES:
        q, k, v = make_qkv(1, H, N, d, dtype, seed=seed, Hkv=Hkv)
        O, lse = mod.attention_fp64(q, k, v, scale, causal, dtype, row_block=2)
        s32 = float(np.float32(scale))
        for h in range(H):
            g = h * Hkv // H
            qf = _decode_independent(q[0, h], dtype)
            kf = _decode_independent(k[0, g], dtype)
            vf = _decode_independent(v[0, g], dtype)
            Ob, lb = brute_force_decimal(qf, kf, vf, s32, causal)
            tol = 1e-13 * (1.0 + abs(s32) * float(np.max(np.abs(qf @ kf.T))))
            _close(O[0, h], Ob, tol * max(1.0, float(np.max(np.abs(vf)))),
                   f"GQA O brute H={H} Hkv={Hkv} head {h}")
            _close(lse[0, h], lb, tol * max(1.0, float(np.max(np.abs(lb)))),
                   f"GQA lse brute H={H} Hkv={Hkv} head {h}")
    # the per-row entry point maps heads the same way
    q, k, v = make_qkv(2, 6, 9, 8, "bf16", seed=35, Hkv=2)
    O, lse = mod.attention_fp64(q, k, v, 0.3, True, "bf16")
    rows = [(0, 0, 3), (1, 5, 8), (0, 2, 0), (1, 3, 6)]
    Or, lr = mod.attention_rows_fp64(q, k, v, 0.3, True, "bf16", rows)
    for t, (b, h, i) in enumerate(rows):
        _close(Or[t], O[b, h, i], 1e-14, "GQA row entry O")
        _close(lr[t], lse[b, h, i], 1e-14, "GQA row entry lse")


def pin_gqa_is_mha_on_repeated_heads(mod):
    """Sharing a key/value head is the same as giving each query head its own
    copy: GQA on [B, Hkv] equals MHA on K, V with each head repeated H/Hkv times."""
    for H, Hkv, causal in [(8, 2, False), (6, 1, True), (4, 4, True)]:
        q, k, v = make_qkv(2, H, 13, 8, "f16", seed=36 + H, Hkv=Hkv)
        O, lse = mod.attention_fp64(q, k, v, 0.35, causal, "f16", row_block=5)
        kr = np.ascontiguousarray(np.repeat(k, H // Hkv, axis=1))
        vr = np.ascontiguousarray(np.repeat(v, H // Hkv, axis=1))
        Or, lr = mod.attention_fp64(q, kr, vr, 0.35, causal, "f16", row_block=5)
        _close(O, Or, 0.0, f"GQA vs repeated heads H={H} Hkv={Hkv}")
        _close(lse, lr, 0.0, f"GQA lse vs repeated heads H={H} Hkv={Hkv}")


def pin_mqa_identical_query_heads(mod):
    """Multi-query attention with every query head the same gives the same
    output in every head, equal to single-head attention."""
    q1, k, v = make_qkv(1, 1, 11, 16, "bf16", seed=40)
    q = np.ascontiguousarray(np.repeat(q1, 5, axis=1))
    for causal in (False, True):
        O, lse = mod.attention_fp64(q, k, v, 0.25, causal, "bf16")
        O1, l1 = mod.attention_fp64(q1, k, v, 0.25, causal, "bf16")
        for h in range(5):
            _close(O[0, h], O1[0, 0], 0.0, "MQA identical heads")
            _close(lse[0, h], l1[0, 0], 0.0, "MQA identical heads lse")


MLA_BRUTE_CASES = [
    # (N, d, dv, dtype, scale, causal, seed): wider queries/keys than values
    (5, 12, 8, "f16", 0.3, True, 51),
    (6, 24, 16, "bf16", 1.0 / math.sqrt(24), False, 52),
    (4, 8, 4, "bf16", -0.6, True, 53),
]


def pin_mla_brute_force(mod):
    """Values narrower than queries and keys (the MLA shape): scores over all d
    columns, outputs with dv columns, against the 50-digit brute force."""
    for N, d, dv, dtype, scale, causal, seed in MLA_BRUTE_CASES:
        q, k, v = make_qkv(1, 2, N, d, dtype, seed=seed, dv=dv)
        O, lse = mod.attention_fp64(q, k, v, scale, causal, dtype, row_block=2)
        if O.shape != (1, 2, N, dv):
            raise AssertionError(f"MLA output shape {O.shape}")
        s32 = float(np.float32(scale))
        for h in range(2):
            qf = _decode_independent(q[0, h], dtype)
            kf = _decode_independent(k[0, h], dtype)
            vf = _decode_independent(v[0, h], dtype)
            Ob, lb = brute_force_decimal(qf, kf, vf, s32, causal)
            tol = 1e-13 * (1.0 + abs(s32) * float(np.max(np.abs(qf @ kf.T))))
            _close(O[0, h], Ob, tol * max(1.0, float(np.max(np.abs(vf)))), f"MLA O d={d} dv={dv}")
            _close(lse[0, h], lb, tol * max(1.0, float(np.max(np.abs(lb)))), f"MLA lse d={d} dv={dv}")


def pin_value_columns_independent(mod):
    """Each output column depends only on the same column of V: splitting V's
    columns into two halves and attending twice gives the two halves of O, and
    lse does not depend on V at all."""
    q, k, v = make_qkv(2, 3, 19, 12, "f16", seed=54, dv=10)
    for causal in (False, True):
        O, lse = mod.attention_fp64(q, k, v, 0.4, causal, "f16", row_block=7)
        O1, l1 = mod.attention_fp64(q, k, np.ascontiguousarray(v[..., :4]), 0.4, causal, "f16")
        O2, l2 = mod.attention_fp64(q, k, np.ascontiguousarray(v[..., 4:]), 0.4, causal, "f16")
        _close(O[..., :4], O1, 1e-14, "V columns 0..3")
        _close(O[..., 4:], O2, 1e-14, "V columns 4..9")
        _close(l1, lse, 0.0, "lse independent of V")
        _close(l2, lse, 0.0, "lse independent of V")


def pin_e4m3_decode(mod):
    """FP8 (OCP E4M3FN) decoding on known codes, and on all 256 codes against
    the library's float8_e4m3fn conversion."""
    codes = np.array([0x38, 0x7E, 0x01, 0x08, 0x80, 0xC5, 0x30, 0x07, 0x77], dtype=np.uint8)
    expect = [1.0, 448.0, 2.0 ** -9, 2.0 ** -6, -0.0, -3.25, 0.5, 7 * 2.0 ** -9, 240.0]
    got = list(mod.decode_fp64(codes, "e4m3"))
    if got != expect or not math.copysign(1.0, got[4]) < 0:
        raise AssertionError(f"e4m3 decode {got} != {expect}")
    if not np.isnan(mod.decode_fp64(np.array([0x7F, 0xFF], dtype=np.uint8), "e4m3")).all():
        raise AssertionError("S.1111.111 must decode to NaN")
    allc = np.arange(256, dtype=np.uint8)
    a = mod.decode_fp64(allc, "e4m3")
    b = _decode_independent(allc, "e4m3")
    same = (a == b) | (np.isnan(a) & np.isnan(b))
    if not same.all():
        raise AssertionError(f"e4m3 decode differs from the library at codes {np.nonzero(~same)[0][:5]}")


def pin_fp8_brute_force(mod):
    """FP8 inputs with per-tensor scales: the oracle equals the 50-digit brute
    force on the scaled decoded values."""
    from seeded_inputs import make_qkv_fp8
    for N, d, scale, causal, seed in [(5, 8, 0.35, True, 61), (7, 16, 0.25, False, 62)]:
        q, k, v, sc = make_qkv_fp8(1, 2, N, d, seed=seed)
        O, lse = mod.attention_fp64(q, k, v, scale, causal, "e4m3", row_block=3, descale=sc)
        s32 = float(np.float32(scale))
        for h in range(2):
            qf = _decode_independent(q[0, h], "e4m3") * float(np.float32(sc[0]))
            kf = _decode_independent(k[0, h], "e4m3") * float(np.float32(sc[1]))
            vf = _decode_independent(v[0, h], "e4m3") * float(np.float32(sc[2]))
            Ob, lb = brute_force_decimal(qf, kf, vf, s32, causal)
            tol = 1e-13 * (1.0 + abs(s32) * float(np.max(np.abs(qf @ kf.T))))
            _close(O[0, h], Ob, tol * max(1.0, float(np.max(np.abs(vf)))), f"FP8 O N={N} d={d}")
            _close(lse[0, h], lb, tol * max(1.0, float(np.max(np.abs(lb)))), f"FP8 lse N={N} d={d}")


ALL_PINS = [
    pin_brute_force,
    pin_zero_query_mean,
    pin_zero_scale_mean,
    pin_softmax_rows,
    pin_shift_invariance,
    pin_constant_value_rows,
    pin_linear_in_v,
    pin_key_permutation,
    pin_single_key,
    pin_causal_special_rows,
    pin_one_hot,
    pin_rows_match_full,
    pin_decode,
    pin_gqa_brute_force,
    pin_gqa_is_mha_on_repeated_heads,
    pin_mqa_identical_query_heads,
    pin_mla_brute_force,
    pin_value_columns_independent,
    pin_e4m3_decode,
    pin_fp8_brute_force,
]
