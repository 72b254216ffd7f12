"""The FP8 parity bound on general inputs, per output element.

Two roundings separate the FP8 kernel from the exact definition (derived in
``tests/test_gpu_fp8.py``'s docstring):

* P is rounded to E4M3 for P.V: relative error at most 2^-4 for a normal
  value, absolute at most 2^-10 in units of the largest weight (half the
  subnormal spacing; the weights are formed against a running maximum no
  larger than the row's true maximum);
* the FP8 matrix core truncates each product in a group of 8 consecutive k
  toward zero to a multiple of 2^(E - 13), E the exponent of the group's
  largest product: at most 7 x 2^-13 of the group's largest product.  On the
  scores that is at most Delta_i = 7 x 2^-13 |scale q_scale k_scale|
  max_j sum_c |q_ic k_jc|, which moves every normalised weight by a factor
  within exp(+-2 Delta_i); on P.V at most 7 x 2^-13 of sum_j P_ij |v_jc|.

So, with P the exact weights and v the real (scaled) values,
    |O - O_ref| <= ((1 + 2^-4) e^(2 Delta_i) (1 + 7 x 2^-13) - 1) sum_j P_ij |v_jc|
                   + 2^-10 e^(2 Delta_i) max_j P_ij sum_{j visible} |v_jc|
                   + fp32 summation terms + half a bf16 ulp of O_ref.

TEST INFRASTRUCTURE: computed from the oracle's own scores and weights.
"""
from __future__ import annotations

import numpy as np

from oracle import decode_fp64, scores_fp64, softmax_rows_fp64
from tests.gpu_util import half_ulp

GROUP_TRUNC = 7 * 2.0 ** -13   # the matrix core's in-group truncation, relative


def summation(N: int) -> float:
    """Relative fp32 error allowance of the two length-N sums (O and l)."""
    return 2 * (N + 128) * 2.0 ** -24 + 1e-5


def rounding_bound(q8_rows: np.ndarray, k8: np.ndarray, v8: np.ndarray, scales, scale: float,
                   causal: bool, rows: np.ndarray, O_ref: np.ndarray) -> np.ndarray:
    """The bound above for some query rows of one head.

    ``q8_rows``: [R, d] E4M3 codes of the rows whose global indices are
    ``rows``; ``k8`` [N, d] and ``v8`` [N, dv]: the codes of the head's
    key/value head; ``O_ref`` [R, dv]: the oracle's outputs of those rows.
    Returns [R, dv].
    """
    sq, sk, sv = (float(np.float32(s)) for s in scales)
    scale64 = float(np.float32(scale))
    cnat = abs(scale64 * sq * sk)
    Kd = decode_fp64(k8, "e4m3")
    Va = np.abs(decode_fp64(v8, "e4m3")) * sv
    Qd = decode_fp64(q8_rows, "e4m3")
    rows = np.asarray(rows)
    # the rows' scores one at a time through the oracle's own functions when
    # they are not consecutive, else as one block
    if rows.size and np.all(np.diff(rows) == 1):
        S = scores_fp64(Qd * sq, Kd * sk, scale64, causal, row0=int(rows[0]))
    else:
        S = np.concatenate([scores_fp64(Qd[t:t + 1] * sq, Kd * sk, scale64, causal,
                                        row0=int(i)) for t, i in enumerate(rows)])
    P, _ = softmax_rows_fp64(S)
    vis = np.isfinite(S)
    # largest sum of |q_c k_c| over the visible keys: the scores' truncation
    absqk = np.where(vis, np.abs(Qd) @ np.abs(Kd).T, 0.0)
    delta = (GROUP_TRUNC + 2.0 ** -20) * cnat * absqk.max(axis=1)
    grow = np.exp(2 * delta)
    pv = P @ Va
    rel = (1 + 2.0 ** -4) * grow * (1 + GROUP_TRUNC) - 1 + summation(k8.shape[0])
    vsum = vis.astype(np.float64) @ Va
    bound = rel[:, None] * pv + 2.0 ** -10 * (grow * P.max(axis=1))[:, None] * vsum
    return bound + half_ulp(O_ref, "bf16")
