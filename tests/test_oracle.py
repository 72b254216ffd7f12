"""The fp64 oracle against its pins, and planted mistakes against the same pins.

CPU only.  A pin failing on the unmodified oracle means the oracle is wrong; a
planted mistake (one small change to the oracle, made here, on the CPU) that no
pin catches means the pins are too weak.
"""
import numpy as np
import pytest

import oracle.softmax_attention as om
from tests import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(om)


# --------------------------------------------------------------------------
# planted mistakes: each replaces one oracle function by a wrong variant
# --------------------------------------------------------------------------
_orig_scores = om.scores_fp64
_orig_softmax = om.softmax_rows_fp64
_orig_decode = om.decode_fp64
_orig_attention = om.attention_fp64


def _scores_no_scale(Q, K, scale, causal, row0=0):
    return _orig_scores(Q, K, 1.0, causal, row0)


def _scores_fixed_scale(Q, K, scale, causal, row0=0):
    return _orig_scores(Q, K, 1.0 / np.sqrt(Q.shape[1]), causal, row0)


def _scores_mask_diagonal(Q, K, scale, causal, row0=0):
    S = (Q @ K.T) * scale
    if causal:
        r = np.arange(row0, row0 + Q.shape[0])[:, None]
        S = np.where(np.arange(K.shape[0])[None, :] >= r, -np.inf, S)
    return S


def _scores_mask_one_late(Q, K, scale, causal, row0=0):
    S = (Q @ K.T) * scale
    if causal:
        r = np.arange(row0, row0 + Q.shape[0])[:, None]
        S = np.where(np.arange(K.shape[0])[None, :] > r + 1, -np.inf, S)
    return S


def _scores_mask_flipped(Q, K, scale, causal, row0=0):
    S = (Q @ K.T) * scale
    if causal:
        r = np.arange(row0, row0 + Q.shape[0])[:, None]
        S = np.where(np.arange(K.shape[0])[None, :] < r, -np.inf, S)
    return S


def _scores_mask_ignores_row0(Q, K, scale, causal, row0=0):
    return _orig_scores(Q, K, scale, causal, 0)


def _scores_keys_reversed(Q, K, scale, causal, row0=0):
    return _orig_scores(Q, K[::-1], scale, causal, row0)


def _scores_transposed(Q, K, scale, causal, row0=0):
    # the "GEMM error" of the paper's Appendix B: operands swapped
    S = (K @ Q.T) * scale
    if causal:
        r = np.arange(row0, row0 + Q.shape[0])[:, None]
        S = np.where(np.arange(K.shape[0])[None, :] > r, -np.inf, S)
    return S


def _scores_scale_in_f32(Q, K, scale, causal, row0=0):
    return _orig_scores(Q, K, float(np.float32(scale) * np.float32(1.0000001)), causal, row0)


def _softmax_no_max(S):
    E = np.exp(S)
    l = E.sum(axis=1, keepdims=True)
    return E / l, np.log(l[:, 0])


def _softmax_lse_without_max(S):
    P, lse = _orig_softmax(S)
    return P, lse - S.max(axis=1)


def _softmax_lse_log2(S):
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    return E / l, m[:, 0] + np.log2(l[:, 0])


def _softmax_unnormalised(S):
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    return E, m[:, 0] + np.log(l[:, 0])


def _softmax_columns_shuffled(S):
    # the "Reshape omission" of the paper's Appendix B: the probabilities reach
    # the second product in a different key order (pairs swapped within blocks)
    P, lse = _orig_softmax(S)
    n = P.shape[1]
    perm = np.arange(n)
    for j in range(0, n - 1, 2):
        perm[j], perm[j + 1] = perm[j + 1], perm[j]
    return P[:, perm], lse


def _decode_bf16_wrong_shift(x, dtype):
    if dtype == "bf16":
        return (x.astype(np.uint32) << np.uint32(15)).view(np.float32).astype(np.float64)
    return _orig_decode(x, dtype)


def _decode_f16_via_bf16(x, dtype):
    if dtype == "f16":
        return (x.view(np.uint16).astype(np.uint32) << np.uint32(16)).view(
            np.float32).astype(np.float64)
    return _orig_decode(x, dtype)


def _attention_last_row_block_dropped(q, k, v, scale, causal, dtype, row_block=256):
    O, lse = _orig_attention(q, k, v, scale, causal, dtype, row_block)
    N = q.shape[2]
    if N > row_block:
        tail = (N - 1) // row_block * row_block
        O[:, :, tail:] = 0.0
    return O, lse


_orig_kv_head = om.kv_head


def _kv_head_modulo(h, H, Hkv):
    # interleaved instead of contiguous groups
    _orig_kv_head(h, H, Hkv)
    return h % Hkv


def _kv_head_first(h, H, Hkv):
    _orig_kv_head(h, H, Hkv)
    return 0


def _scores_truncated_to_value_width(Q, K, scale, causal, row0=0):
    # scores over only the first 3/4 of the head (as if sized by the value width)
    w = max(1, (Q.shape[1] * 3) // 4)
    return _orig_scores(Q[:, :w], K[:, :w], scale, causal, row0)


def _decode_e4m3_bias8(x, dtype):
    # the exponent bias of the other FP8 variant (E4M3 with bias 8)
    if dtype == "e4m3":
        return _orig_decode(x, dtype) / 2.0
    return _orig_decode(x, dtype)


def _attention_ignores_value_scale(q, k, v, scale, causal, dtype, row_block=256, descale=None):
    if descale is not None:
        descale = (descale[0], descale[1], 1.0)
    return _orig_attention(q, k, v, scale, causal, dtype, row_block, descale)


MUTANTS = {
    "scores_no_scale": ("scores_fp64", _scores_no_scale),
    "scores_fixed_scale": ("scores_fp64", _scores_fixed_scale),
    "scores_mask_diagonal": ("scores_fp64", _scores_mask_diagonal),
    "scores_mask_one_late": ("scores_fp64", _scores_mask_one_late),
    "scores_mask_flipped": ("scores_fp64", _scores_mask_flipped),
    "scores_mask_ignores_row0": ("scores_fp64", _scores_mask_ignores_row0),
    "scores_keys_reversed": ("scores_fp64", _scores_keys_reversed),
    "scores_transposed": ("scores_fp64", _scores_transposed),
    "scores_scale_off_by_1e-7": ("scores_fp64", _scores_scale_in_f32),
    "softmax_no_max": ("softmax_rows_fp64", _softmax_no_max),
    "softmax_lse_without_max": ("softmax_rows_fp64", _softmax_lse_without_max),
    "softmax_lse_log2": ("softmax_rows_fp64", _softmax_lse_log2),
    "softmax_unnormalised": ("softmax_rows_fp64", _softmax_unnormalised),
    "softmax_columns_shuffled": ("softmax_rows_fp64", _softmax_columns_shuffled),
    "decode_bf16_wrong_shift": ("decode_fp64", _decode_bf16_wrong_shift),
    "decode_f16_as_bf16": ("decode_fp64", _decode_f16_via_bf16),
    "attention_drops_tail_rows": ("attention_fp64", _attention_last_row_block_dropped),
    "kv_head_interleaved": ("kv_head", _kv_head_modulo),
    "kv_head_always_first": ("kv_head", _kv_head_first),
    "scores_truncated": ("scores_fp64", _scores_truncated_to_value_width),
    "decode_e4m3_bias8": ("decode_fp64", _decode_e4m3_bias8),
    "attention_ignores_value_scale": ("attention_fp64", _attention_ignores_value_scale),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(om, attr, fn)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(om)
        except (AssertionError, ValueError, FloatingPointError, TypeError) as e:
            caught.append((pin.__name__, str(e)[:80]))
    assert caught, f"planted mistake {name!r} passes every pin"
