"""fp64 CPU oracle for the fused attention forward.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or call it. The product path
(``paper_2506_12355_amd``) never imports it, and it imports nothing from the
product path.
"""
from .softmax_attention import (  # noqa: F401
    attention_fp64,
    attention_rows_fp64,
    decode_fp64,
    kv_head,
    scores_fp64,
    softmax_rows_fp64,
)
