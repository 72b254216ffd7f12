"""The C-ABI boundary without a GPU: the library loads, exports every declared
symbol, and rejects every invalid argument with its documented status before
touching the device.

Every call here carries at least one invalid argument, so nothing is ever
enqueued (the library validates on the host before any HIP call).
"""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2506_12355_amd as qa
from paper_2506_12355_amd import build as qbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(qa.LIB_PATH):
        qbuild.build()
    return qa.load_library()


def _declared_functions():
    names = []
    inc = os.path.join(ROOT, "include")
    for fn in sorted(os.listdir(inc)):
        if fn.endswith(".h"):
            text = open(os.path.join(inc, fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b(qm_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_entry_points():
    assert {"qm_attn_fwd", "qm_attn_fwd_gqa", "qm_attn_fwd_mla", "qm_attn_fwd_fp8",
            "qm_attn_fwd_layout", "qm_attn_fwd_fp8_layout", "qm_attn_set_tile_rows",
            "qm_attn_strerror"} <= set(_declared_functions())


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", qa.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in _declared_functions():
        assert name in exported, f"{name} declared in include/ but not exported"
        assert hasattr(lib, name)


def test_library_has_no_undefined_kernel_symbols(lib):
    """Every kernel's host launch stub is defined in the library itself."""
    out = subprocess.run(["nm", "-D", "--undefined-only", qa.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    missing = [line.split()[-1] for line in out.splitlines() if "qm" in line]
    assert not missing, f"undefined symbols from the library's own code: {missing}"


# fake, well-separated, 256-byte aligned device addresses: never dereferenced
GIB = 1 << 30
Q, K, V, O, L = (GIB * i for i in range(1, 6))
GOOD = dict(q=Q, k=K, v=V, o=O, lse=L, B=1, H=2, N=128, d=64, scale=0.125, causal=0,
            stream=None, dtype=qa.QM_F16)


def call(**over):
    a = dict(GOOD)
    a.update(over)
    return qa.qm_attn_fwd(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"], a["N"],
                          a["d"], a["scale"], a["causal"], a["stream"], a["dtype"])


@pytest.mark.parametrize("over,status", [
    (dict(q=None), qa.QM_ERR_NULL),
    (dict(k=None), qa.QM_ERR_NULL),
    (dict(v=None), qa.QM_ERR_NULL),
    (dict(o=None), qa.QM_ERR_NULL),
    (dict(lse=None), qa.QM_ERR_NULL),
    (dict(B=0), qa.QM_ERR_SHAPE),
    (dict(H=-1), qa.QM_ERR_SHAPE),
    (dict(N=0), qa.QM_ERR_SHAPE),
    (dict(N=1 << 24, d=128), qa.QM_ERR_SHAPE),            # one head's slab >= 2^31 elements
    (dict(N=(1 << 31) - 1), qa.QM_ERR_SHAPE),             # N + 256 would overflow an int
    (dict(N=(1 << 31) - 200, d=128), qa.QM_ERR_SHAPE),
    (dict(B=1 << 30, H=1 << 30, N=1 << 16, d=64), qa.QM_ERR_SHAPE),
    (dict(d=96), qa.QM_ERR_HEADDIM),
    (dict(d=256), qa.QM_ERR_HEADDIM),
    (dict(d=0), qa.QM_ERR_HEADDIM),
    (dict(dtype=2), qa.QM_ERR_DTYPE),
    (dict(dtype=-1), qa.QM_ERR_DTYPE),
    (dict(scale=float("inf")), qa.QM_ERR_SCALE),
    (dict(scale=float("-inf")), qa.QM_ERR_SCALE),
    (dict(scale=float("nan")), qa.QM_ERR_SCALE),
    (dict(scale=1e39), qa.QM_ERR_SCALE),                  # overflows float32 to inf
    (dict(causal=2), qa.QM_ERR_CAUSAL),
    (dict(causal=-1), qa.QM_ERR_CAUSAL),
    (dict(o=Q), qa.QM_ERR_ALIAS),
    (dict(o=K + 4096), qa.QM_ERR_ALIAS),
    (dict(lse=V + 256), qa.QM_ERR_ALIAS),
    (dict(lse=O + 16), qa.QM_ERR_ALIAS),
    (dict(o=L - 1024), qa.QM_ERR_ALIAS),                  # o's tail runs into lse
    (dict(q=Q + 8), qa.QM_ERR_UNSUPPORTED),
    (dict(o=O + 2), qa.QM_ERR_UNSUPPORTED),
    (dict(lse=L + 4), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_invalid_arguments_are_rejected(lib, over, status):
    assert call(**over) == status


def call_gqa(Hkv, **over):
    a = dict(GOOD)
    a.update(over)
    return qa.qm_attn_fwd_gqa(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"], Hkv,
                              a["N"], a["d"], a["scale"], a["causal"], a["stream"], a["dtype"])


@pytest.mark.parametrize("H,Hkv,over,status", [
    (8, 0, {}, qa.QM_ERR_SHAPE),
    (8, -2, {}, qa.QM_ERR_SHAPE),
    (8, 16, {}, qa.QM_ERR_SHAPE),                       # more key/value heads than query heads
    (8, 3, {}, qa.QM_ERR_SHAPE),                        # does not divide H
    (6, 4, {}, qa.QM_ERR_SHAPE),
    (8, 2, dict(k=None), qa.QM_ERR_NULL),
    (8, 2, dict(d=96), qa.QM_ERR_HEADDIM),
    (8, 2, dict(dtype=5), qa.QM_ERR_DTYPE),
    (8, 2, dict(scale=float("nan")), qa.QM_ERR_SCALE),
    (8, 2, dict(causal=3), qa.QM_ERR_CAUSAL),
    (8, 2, dict(o=K + 16 * 1024), qa.QM_ERR_ALIAS),       # inside k's 2-head extent
    (8, 2, dict(lse=V + 16), qa.QM_ERR_ALIAS),
    (8, 2, dict(v=V + 8), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_gqa_invalid_arguments_are_rejected(lib, H, Hkv, over, status):
    assert call_gqa(Hkv, H=H, **over) == status


def test_gqa_alias_extent_follows_kv_heads(lib):
    """k and v hold Hkv heads, so o may start right after k's shorter extent.
    A misaligned lse (checked after the alias rules) keeps anything from being
    enqueued either way."""
    kv_bytes = 1 * 2 * 128 * 64 * 2          # B=1, Hkv=2, N=128, d=64, 16-bit
    assert call_gqa(2, H=8, o=K + kv_bytes, lse=L + 4) == qa.QM_ERR_UNSUPPORTED
    assert call_gqa(8, H=8, o=K + kv_bytes, lse=L + 4) == qa.QM_ERR_ALIAS


def call_mla(d_qk, d_v, **over):
    a = dict(GOOD)
    a.update(over)
    return qa.qm_attn_fwd_mla(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"], a["N"],
                              d_qk, d_v, a["scale"], a["causal"], a["stream"], a["dtype"])


@pytest.mark.parametrize("d_qk,d_v,over,status", [
    (192, 192, {}, qa.QM_ERR_HEADDIM),
    (128, 64, {}, qa.QM_ERR_HEADDIM),
    (192, 64, {}, qa.QM_ERR_HEADDIM),
    (256, 128, {}, qa.QM_ERR_HEADDIM),
    (64, 128, {}, qa.QM_ERR_HEADDIM),
    (192, 128, dict(v=None), qa.QM_ERR_NULL),
    (192, 128, dict(N=0), qa.QM_ERR_SHAPE),
    (192, 128, dict(N=(1 << 31) // 192 - 100), qa.QM_ERR_SHAPE),   # one q/k head >= 2^31 elements
    (192, 128, dict(dtype=3), qa.QM_ERR_DTYPE),
    (192, 128, dict(scale=float("inf")), qa.QM_ERR_SCALE),
    (192, 128, dict(causal=7), qa.QM_ERR_CAUSAL),
    # B=1, H=2, N=128: q and k span 96 KiB at d_qk = 192, v 64 KiB at d_v = 128
    (192, 128, dict(o=Q + 80 * 1024), qa.QM_ERR_ALIAS),          # inside q's wider extent
    (192, 128, dict(lse=K + 90 * 1024), qa.QM_ERR_ALIAS),
    (192, 128, dict(o=O + 8), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_mla_invalid_arguments_are_rejected(lib, d_qk, d_v, over, status):
    assert call_mla(d_qk, d_v, **over) == status


def test_plain_entry_rejects_the_mla_head(lib):
    assert call(d=192) == qa.QM_ERR_HEADDIM


def call_layout(layout, Hkv=None, d_v=None, **over):
    a = dict(GOOD)
    a.update(over)
    return qa.qm_attn_fwd_layout(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"],
                                 a["H"] if Hkv is None else Hkv, a["N"], a["d"],
                                 a["d"] if d_v is None else d_v, a["scale"], a["causal"],
                                 a["stream"], a["dtype"], layout)


@pytest.mark.parametrize("layout,kw,status", [
    (2, {}, qa.QM_ERR_LAYOUT),
    (-1, {}, qa.QM_ERR_LAYOUT),
    (qa.QM_BNHD, dict(d=192, d_v=128), qa.QM_ERR_LAYOUT),      # 192-wide keys: [B][H][N][d] only
    # a head's rows 64 heads apart: (N + 256) * 64 * 128 * 2 bytes overflow 32 bits
    (qa.QM_BNHD, dict(N=1 << 20, H=64, d=128), qa.QM_ERR_SHAPE),
    (qa.QM_BNHD, dict(N=(1 << 31) - 1), qa.QM_ERR_SHAPE),     # N + 256 would overflow an int
    (qa.QM_BNHD, dict(N=1 << 20, H=64, d=128, q=None), qa.QM_ERR_NULL),   # NULL comes first
    (qa.QM_BHND, dict(d=96), qa.QM_ERR_HEADDIM),
    (qa.QM_BNHD, dict(causal=3), qa.QM_ERR_CAUSAL),
    (qa.QM_BNHD, dict(Hkv=3), qa.QM_ERR_SHAPE),                # 3 does not divide H = 2
    (qa.QM_BNHD, dict(o=Q + 2), qa.QM_ERR_ALIAS),
    (qa.QM_BNHD, dict(k=K + 8), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_layout_entry_rejects_invalid_arguments(lib, layout, kw, status):
    assert call_layout(layout, **kw) == status


def test_layout_error_text(lib):
    assert "QM_BNHD" in qa.strerror(qa.QM_ERR_LAYOUT)


def call_fp8(qs=0.01, ks=0.01, vs=0.01, **over):
    a = dict(GOOD)
    a.update(over)
    return qa.qm_attn_fwd_fp8(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"], a["N"],
                              a["d"], qs, ks, vs, a["scale"], a["causal"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(d=64), qa.QM_ERR_HEADDIM),                    # FP8 runs at d = 128 only
    (dict(d=192), qa.QM_ERR_HEADDIM),
    (dict(d=128, q=None), qa.QM_ERR_NULL),
    (dict(d=128, N=0), qa.QM_ERR_SHAPE),
    (dict(d=128, qs=float("inf")), qa.QM_ERR_SCALE),
    (dict(d=128, ks=float("nan")), qa.QM_ERR_SCALE),
    (dict(d=128, vs=float("-inf")), qa.QM_ERR_SCALE),
    (dict(d=128, scale=float("nan")), qa.QM_ERR_SCALE),
    (dict(d=128, qs=3e38, ks=3e38, lse=L + 4), qa.QM_ERR_UNSUPPORTED),   # alignment comes first
    (dict(d=128, qs=3e38, ks=3e38), qa.QM_ERR_SCALE),    # the combined scale overflows
    (dict(d=128, causal=2), qa.QM_ERR_CAUSAL),
    # B=1, H=2, N=128, d=128: q, k, v span 32 KiB of one-byte codes, o 64 KiB of bf16
    (dict(d=128, o=Q + 16 * 1024), qa.QM_ERR_ALIAS),
    (dict(d=128, lse=V + 8 * 1024), qa.QM_ERR_ALIAS),
    (dict(d=128, k=K + 8), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_fp8_invalid_arguments_are_rejected(lib, kw, status):
    kw = dict(kw)
    qs, ks, vs = kw.pop("qs", 0.01), kw.pop("ks", 0.01), kw.pop("vs", 0.01)
    assert call_fp8(qs, ks, vs, **kw) == status


def call_fp8_layout(layout, Hkv=None, qs=0.01, ks=0.01, vs=0.01, **over):
    a = dict(GOOD, d=128)
    a.update(over)
    return qa.qm_attn_fwd_fp8_layout(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"],
                                     a["H"] if Hkv is None else Hkv, a["N"], a["d"], qs, ks, vs,
                                     a["scale"], a["causal"], a["stream"], layout)


@pytest.mark.parametrize("layout,kw,status", [
    (2, {}, qa.QM_ERR_LAYOUT),
    (-1, dict(Hkv=1), qa.QM_ERR_LAYOUT),
    (qa.QM_BNHD, dict(d=64), qa.QM_ERR_HEADDIM),          # FP8 runs at d = 128 only
    (qa.QM_BHND, dict(d=192), qa.QM_ERR_HEADDIM),
    (qa.QM_BHND, dict(Hkv=0), qa.QM_ERR_SHAPE),
    (qa.QM_BNHD, dict(Hkv=3), qa.QM_ERR_SHAPE),           # 3 does not divide H = 2
    (qa.QM_BNHD, dict(Hkv=4), qa.QM_ERR_SHAPE),           # more key/value heads than query heads
    (qa.QM_BNHD, dict(v=None), qa.QM_ERR_NULL),
    (qa.QM_BNHD, dict(vs=float("nan")), qa.QM_ERR_SCALE),
    (qa.QM_BHND, dict(Hkv=1, qs=3e38, ks=3e38), qa.QM_ERR_SCALE),
    (qa.QM_BNHD, dict(causal=5), qa.QM_ERR_CAUSAL),
    # B=1, H=2, Hkv=1, N=128, d=128: k spans 16 KiB of one-byte codes
    (qa.QM_BHND, dict(Hkv=1, o=K + 8 * 1024), qa.QM_ERR_ALIAS),
    (qa.QM_BNHD, dict(Hkv=1, lse=L + 4), qa.QM_ERR_UNSUPPORTED),
], ids=lambda x: str(x))
def test_fp8_layout_entry_rejects_invalid_arguments(lib, layout, kw, status):
    kw = dict(kw)
    Hkv = kw.pop("Hkv", None)
    assert call_fp8_layout(layout, Hkv, **kw) == status


def test_fp8_layout_row_bound_counts_one_byte_codes(lib):
    """[B][N][H][d] rows of one-byte codes are half as wide as 16-bit ones, so
    N = 2^18 with 64 heads of 128 fits the kernels' 32-bit offsets in FP8
    (the call gets as far as the alignment check) but not in bf16."""
    T = 1 << 40
    big = dict(q=T, k=2 * T, v=3 * T, o=4 * T, lse=5 * T + 4, N=1 << 18, H=64, d=128)
    assert call_fp8_layout(qa.QM_BNHD, **big) == qa.QM_ERR_UNSUPPORTED
    assert call_fp8_layout(qa.QM_BNHD, **dict(big, N=1 << 19)) == qa.QM_ERR_SHAPE
    assert call_layout(qa.QM_BNHD, **dict(big, dtype=qa.QM_BF16)) == qa.QM_ERR_SHAPE
    assert call_layout(qa.QM_BHND, **dict(big, dtype=qa.QM_BF16)) == qa.QM_ERR_UNSUPPORTED


def test_tile_rows_control_accepts_only_its_values(lib):
    try:
        for rows in (1, 64, 192, 512, -128):
            assert lib.qm_attn_set_tile_rows(rows) == qa.QM_ERR_TILE
        for rows in (128, 256, 0):
            assert lib.qm_attn_set_tile_rows(rows) == qa.QM_OK
        with pytest.raises(qa.QmAttnError) as e:
            qa.set_tile_rows(100)
        assert e.value.status == qa.QM_ERR_TILE
        assert "128 or 256" in qa.strerror(qa.QM_ERR_TILE)
    finally:
        lib.qm_attn_set_tile_rows(0)


def test_16bit_entries_reject_the_fp8_code(lib):
    assert call(dtype=2) == qa.QM_ERR_DTYPE
    assert call_gqa(1, H=2, dtype=2) == qa.QM_ERR_DTYPE
    assert call_mla(128, 128, dtype=2) == qa.QM_ERR_DTYPE
    assert call_layout(qa.QM_BHND, dtype=2) == qa.QM_ERR_DTYPE


def test_inputs_may_alias_each_other(lib):
    # q = k = v is legal (read-only); the call still fails on the bad dtype, which
    # is checked after the alias rules, so no kernel is ever enqueued here
    assert call(k=Q, v=Q, dtype=7) == qa.QM_ERR_DTYPE


def test_strerror(lib):
    codes = [qa.QM_OK, qa.QM_ERR_NULL, qa.QM_ERR_SHAPE, qa.QM_ERR_HEADDIM, qa.QM_ERR_DTYPE,
             qa.QM_ERR_SCALE, qa.QM_ERR_ALIAS, qa.QM_ERR_CAUSAL, qa.QM_ERR_LAUNCH,
             qa.QM_ERR_UNSUPPORTED, qa.QM_ERR_LAYOUT, qa.QM_ERR_TILE]
    msgs = [qa.strerror(c) for c in codes]
    assert len(set(msgs)) == len(codes)
    assert qa.strerror(12345) == "unknown status"


def test_python_wrapper_rejects_host_tensors(lib):
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 1, 4, 64, dtype=torch.float16)
    with pytest.raises(ValueError):
        qa.fwd(x, x, x)
    with pytest.raises(ValueError):
        qa.fwd(x[0], x[0], x[0])


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    import paper_2506_12355_amd.binding as b
    monkeypatch.setattr(b, "_lib", None)
    with pytest.raises(RuntimeError, match="has not been built"):
        b.load_library(str(tmp_path / "libqm_attn.so"))


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2506_12355_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, fn)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle", text, re.M), fn
                assert "softmax_attention" not in text, fn


def test_c_client_builds_and_checks_buffer_sizes(lib):
    """The plain-C client of the C ABI (driven on the GPU by
    test_gpu_c_client.py) compiles with gcc against include/qm_attn.h, links
    the library, and refuses a buffer smaller than its shape before any HIP
    call."""
    import ctypes
    import numpy as np
    from tests import build_c_client, test_gpu_c_client as tc
    if not os.path.exists(build_c_client.OUT):
        build_c_client.build()
    client = tc.load_client()
    x = np.zeros(16, dtype=np.uint16)
    msg = ctypes.create_string_buffer(128)
    st = client.qmc_run(0, x.ctypes.data, x.nbytes, x.ctypes.data, x.nbytes, x.ctypes.data,
                        x.nbytes, x.ctypes.data, x.nbytes, x.ctypes.data, x.nbytes,
                        1, 2, 2, 128, 64, 64, 0.125, 0, 0, 0, 1.0, 1.0, 1.0, msg, len(msg))
    assert st == -100 and b"smaller" in msg.value
