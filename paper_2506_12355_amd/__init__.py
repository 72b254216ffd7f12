"""MI355X-native fused attention forward: gfx950 HIP kernels behind a C ABI.

``fwd(q, k, v, causal, scale)`` computes softmax(mask(scale * Q K^T)) V and the
per-row log-sum-exp for [B, H, N, d] fp16/bf16 tensors on one GPU; k and v may
have fewer heads than q (grouped-query and multi-query attention), and v a
narrower head than q and k (the MLA shape, 192/128).  ``fwd_fp8`` takes FP8
(E4M3) inputs with per-tensor scales, also with fewer key/value heads; ``fwd(..., layout="bnhd")`` takes
[B, N, heads, d] tensors.  The
operation and its arguments are documented in ``include/qm_attn.h``.
"""
from .binding import (  # noqa: F401
    DEBUG_LIB_PATH,
    LIB_PATH,
    QM_BF16,
    QM_BHND,
    QM_BNHD,
    QM_ERR_ALIAS,
    QM_ERR_CAUSAL,
    QM_ERR_DTYPE,
    QM_ERR_HEADDIM,
    QM_ERR_LAUNCH,
    QM_ERR_LAYOUT,
    QM_ERR_NULL,
    QM_ERR_SCALE,
    QM_ERR_SHAPE,
    QM_ERR_TILE,
    QM_ERR_UNSUPPORTED,
    QM_F16,
    QM_OK,
    QmAttnError,
    fwd,
    fwd_fp8,
    load_library,
    open_library,
    qm_attn_fwd,
    qm_attn_fwd_fp8,
    qm_attn_fwd_fp8_layout,
    qm_attn_fwd_gqa,
    qm_attn_fwd_layout,
    qm_attn_fwd_mla,
    set_tile_rows,
    strerror,
)
