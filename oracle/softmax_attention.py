"""Plain fp64 CPU oracle for softmax attention (the operator the fused kernel computes).

TEST INFRASTRUCTURE ONLY: used by ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py``; never by the product path.

What it follows
---------------
The paper states the problem in its Background, subsection "Attention
Operators and acceleration": with Q, K, V holding N tokens of dimension d,
Attention(Q, K, V) = Softmax(Mask(Q K^T / sqrt(d))) V, evaluated independently
for every (batch, head).  A FlashAttention-style kernel reaches exactly this
value (up to rounding order); it only reorders the work.  So this oracle is the
definition written out, per (batch, head):

1. decode the 16-bit inputs to fp64 exactly (:func:`decode_fp64`);
2. scores s_ij = scale * (q_i . k_j) in fp64 (:func:`scores_fp64`); the scale
   is a parameter, taken as the same fp32 value the kernel receives;
3. mask: with ``causal``, key j is visible to query i iff j <= i; a masked
   score is -inf (the paper leaves "Mask" undefined; the Evaluation section
   only names "causal masks");
4. row softmax with the row maximum subtracted (the paper's Appendix B
   listing computes the softmax "with Smax and Ssum"), giving P and the
   natural-log log-sum-exp lse_i = m_i + ln(sum_j exp(s_ij - m_i))
   (:func:`softmax_rows_fp64`);
5. O = P V (:func:`attention_fp64`).

Grouped-query and multi-query attention (named beside multi-head attention in
the same Background subsection, and evaluated in the Evaluation section): H
query heads share Hkv key/value heads.  The paper does not spell out the
grouping; the reading here is the contiguous one, query head h using
key/value head h // (H / Hkv) (:func:`kv_head`).  Each query head is then
exactly the definition above with its group's K and V.

Queries are processed in independent row blocks only to bound memory; each
row's value is the definition's.  There is no online rescaling, no key
blocking and no fusion.

Readings where the paper is silent: the head layout is [B, H, N, d]; lse is
the natural logarithm; the scale is applied to the exact dot product, never to
16-bit Q.  FP8 inputs (OCP E4M3 codes) come with per-tensor scale factors:
the real tensors are the scaled decoded values, and the definition applies to
those.  Values may have their own head dimension d_v (the MLA shape the
paper evaluates: queries and keys 128 + 64 wide, values 128): the scores use
all d columns of Q and K, the output has d_v columns.

Pins: ``tests/test_oracle.py`` checks every function here against a
high-precision brute force, closed forms, invariants and special cases, and
shows that planted mistakes fail those pins.
"""
from __future__ import annotations

import numpy as np

_F64_DTYPES = ("f16", "bf16", "e4m3", "f64")


def _e4m3_value(c: int) -> float:
    """OCP E4M3FN code c: sign, 4 exponent bits with bias 7, 3 mantissa bits;
    exponent field 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; no infinity."""
    sign = -1.0 if c & 0x80 else 1.0
    e, m = (c >> 3) & 0xF, c & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


_E4M3_TABLE = np.array([_e4m3_value(c) for c in range(256)], dtype=np.float64)


def decode_fp64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored inputs to fp64, exactly.

    ``f16``: ``numpy.float16`` values; ``bf16``: ``uint16`` bit patterns (the
    top half of an IEEE fp32); ``e4m3``: ``uint8`` OCP E4M3FN codes (FP8);
    ``f64``: already fp64 (used by the pins).
    """
    if dtype == "f16":
        if x.dtype != np.float16:
            raise TypeError("f16 input must be numpy.float16")
        return x.astype(np.float64)
    if dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 input must be uint16 bit patterns")
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "e4m3":
        if x.dtype != np.uint8:
            raise TypeError("e4m3 input must be uint8 codes")
        return _E4M3_TABLE[x]
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(f"unknown dtype {dtype!r}; expected one of {_F64_DTYPES}")


def _descale(descale):
    if descale is None:
        return 1.0, 1.0, 1.0
    return tuple(float(np.float32(t)) for t in descale)


def kv_head(h: int, H: int, Hkv: int) -> int:
    """Key/value head read by query head ``h`` when H query heads share Hkv."""
    if Hkv < 1 or H % Hkv != 0:
        raise ValueError(f"{Hkv} key/value heads cannot be shared by {H} query heads")
    return h // (H // Hkv)


def scores_fp64(Q: np.ndarray, K: np.ndarray, scale: float, causal: bool,
                row0: int = 0) -> np.ndarray:
    """Masked scaled scores for one (batch, head).

    ``Q``: [R, d] fp64 queries whose global row indices are row0 .. row0+R-1;
    ``K``: [Nk, d] fp64 keys.  Returns S [R, Nk] with s_ij = scale * (q_i . k_j)
    and -inf where the causal mask hides key j from query i (j > i).
    """
    S = (Q @ K.T) * np.float64(scale)
    if causal:
        rows = np.arange(row0, row0 + Q.shape[0])[:, None]
        cols = np.arange(K.shape[0])[None, :]
        S = np.where(cols > rows, -np.inf, S)
    return S


def softmax_rows_fp64(S: np.ndarray):
    """Row softmax of masked scores with the row maximum subtracted.

    Returns (P, lse): P [R, Nk] with rows summing to 1, and the natural-log
    log-sum-exp lse [R].  Every row must have at least one finite score (a
    causal square mask always leaves key 0 visible).
    """
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    P = E / l
    lse = m[:, 0] + np.log(l[:, 0])
    return P, lse


def attention_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                   causal: bool, dtype: str, row_block: int = 256, descale=None):
    """Exact attention forward for every (batch, head): q [B, H, N, d], k
    [B, Hkv, N, d] and v [B, Hkv, N, dv] with Hkv dividing H (Hkv = H:
    multi-head attention).

    ``descale``: optional per-tensor factors (sq, sk, sv), taken as float32
    values: the real tensors are sq*Q, sk*K and sv*V (FP8 inputs).

    Returns (O [B, H, N, dv] fp64, lse [B, H, N] fp64).
    """
    B, H, N, d = q.shape
    sq, sk, sv = _descale(descale)
    Hkv = k.shape[1] if k.ndim == 4 else -1
    dv = v.shape[-1] if v.ndim == 4 else -1
    if k.shape != (B, Hkv, N, d) or v.shape != (B, Hkv, N, dv):
        raise ValueError("k must be [B, Hkv, N, d] and v [B, Hkv, N, dv] with q's B, N, d")
    scale64 = float(np.float32(scale)) if dtype != "f64" else float(scale)
    O = np.empty((B, H, N, dv), dtype=np.float64)
    lse = np.empty((B, H, N), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            K = decode_fp64(k[b, kv_head(h, H, Hkv)], dtype) * sk
            V = decode_fp64(v[b, kv_head(h, H, Hkv)], dtype) * sv
            for r0 in range(0, N, row_block):
                r1 = min(N, r0 + row_block)
                Q = decode_fp64(q[b, h, r0:r1], dtype) * sq
                S = scores_fp64(Q, K, scale64, causal, row0=r0)
                P, lse_blk = softmax_rows_fp64(S)
                O[b, h, r0:r1] = P @ V
                lse[b, h, r0:r1] = lse_blk
    return O, lse


def attention_rows_fp64(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                        causal: bool, dtype: str, rows, descale=None):
    """Exact attention output for selected rows only.

    ``rows``: iterable of (b, h, i).  Returns (O [R, dv] fp64, lse [R] fp64) in
    the order given.  Used where the full output is too large for the CPU:
    each selected row is the definition's value, computed from that row's
    query against all of its (visible) keys.
    """
    rows = [tuple(int(t) for t in r) for r in rows]
    sq, sk, sv = _descale(descale)
    H = q.shape[1]
    Hkv = k.shape[1]
    O = np.empty((len(rows), v.shape[-1]), dtype=np.float64)
    lse = np.empty(len(rows), dtype=np.float64)
    scale64 = float(np.float32(scale)) if dtype != "f64" else float(scale)
    by_head = {}
    for idx, (b, h, i) in enumerate(rows):
        by_head.setdefault((b, h), []).append((idx, i))
    for (b, h), items in by_head.items():
        K = decode_fp64(k[b, kv_head(h, H, Hkv)], dtype) * sk
        V = decode_fp64(v[b, kv_head(h, H, Hkv)], dtype) * sv
        for idx, i in items:
            Q = decode_fp64(q[b, h, i:i + 1], dtype) * sq
            S = scores_fp64(Q, K, scale64, causal, row0=i)
            P, lse_row = softmax_rows_fp64(S)
            O[idx] = (P @ V)[0]
            lse[idx] = lse_row[0]
    return O, lse
