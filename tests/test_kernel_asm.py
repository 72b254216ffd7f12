"""The gfx950 kernels as compiled (CPU only: hipcc cross-compiles the device code).

* every direct HBM -> LDS load is clear of the VALU-write-SGPR hazard its
  inline assembly must resolve by itself;
* no packed fp32 instruction appears in device code;
* no kernel spills VGPRs or uses scratch memory.
"""
from __future__ import annotations

import os
import re
import subprocess

import pytest

from paper_2506_12355_amd import build as qbuild
from tests.asm_hazards import dma_sgpr_hazards, instructions, is_direct_load


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    try:
        cc = qbuild.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "attn.s")
    flags = [f for f in qbuild.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    cmd = ([cc] + flags + ["--cuda-device-only", "-S", "-I", qbuild.INCLUDE, "-I", qbuild.CSRC,
                           "-o", out, os.path.join(qbuild.CSRC, "attn_fwd_gfx950.hip")])
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return open(out).read()


def _kernels(text):
    """name -> instruction list, one per kernel instance."""
    out = {}
    for m in re.finditer(r"^(_Z\w*attn_fwd_kernel\w*):\s*(?:;.*)?$", text, flags=re.M):
        end = text.index(".Lfunc_end", m.end())   # a kernel may hold several s_endpgm
        out[m.group(1)] = instructions(text[m.end():end])
    return out


N_INSTANCES = 24   # eight waves: 16-bit (64,64), (128,128), (192,128) x dtype x mask and FP8
                   # (128,128) x mask; four waves: the same without (192,128)


def test_all_instances_compiled(asm):
    names = list(_kernels(asm))
    assert len(names) == N_INSTANCES
    assert sum("ELi8EEEv" in n for n in names) == 14
    assert sum("ELi4EEEv" in n for n in names) == 10


def test_direct_loads_have_no_sgpr_hazard(asm):
    for name, insts in _kernels(asm).items():
        assert any(is_direct_load(i) for i in insts), name
        bad = dma_sgpr_hazards(insts)
        assert not bad, f"{name}: {bad[:3]}"


def test_no_packed_fp32(asm):
    for name, insts in _kernels(asm).items():
        bad = [i for i in insts if re.match(r"v_pk_(add|mul|fma|mov)_f32", i)]
        assert not bad, f"{name}: {bad[:3]}"


def test_fp8_products_use_the_unscaled_mfma(asm):
    """The FP8 instances pass zero block-scale operands, which the compiler maps
    to the unscaled 32x32x64 instruction; a block-scaled form with scale code 0
    would multiply every product by 2^-254."""
    fp8 = {n: i for n, i in _kernels(asm).items() if "ELi2ELb" in n}   # dtype 2: FP8
    assert len(fp8) == 4   # two masks, two workgroup sizes
    for name, insts in fp8.items():
        ops = [i.split()[0] for i in insts]
        assert ops.count("v_mfma_f32_32x32x64_f8f6f4") >= 8, name
        assert not any(o.startswith("v_mfma_scale") for o in ops), name


def test_no_spills_or_scratch(asm):
    spills = [int(x) for x in re.findall(r"\.vgpr_spill_count:\s+(\d+)", asm)]
    scratch = [int(x) for x in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", asm)]
    assert len(spills) == N_INSTANCES and max(spills) == 0
    assert len(scratch) == N_INSTANCES and max(scratch) == 0


def test_checker_sees_a_planted_hazard():
    """The hazard scan itself: a VALU write of a descriptor SGPR two instructions
    before a direct load is reported; five wait states in between clear it."""
    bad = ["v_readlane_b32 s5, v243, 3", "s_mov_b32 s0, 0",
           "buffer_load_dwordx4 v1, s[4:7], 0 offen lds"]
    assert len(dma_sgpr_hazards(bad)) == 1
    ok = ["v_readlane_b32 s5, v243, 3", "s_nop 4", "buffer_load_dwordx4 v1, s[4:7], 0 offen lds"]
    assert dma_sgpr_hazards(ok) == []
    other = ["v_readlane_b32 s9, v243, 3", "buffer_load_dwordx4 v1, s[4:7], 0 offen lds"]
    assert dma_sgpr_hazards(other) == []


def test_register_budgets_admit_the_planned_occupancy(asm):
    """Two waves per SIMD for every instance (at most 256 VGPRs), and three
    four-wave workgroups per CU at d = 64 (at most 168 VGPRs: three waves of
    a SIMD's 512)."""
    names = re.findall(r"\.name:\s+(\S*attn_fwd_kernel\S*)", asm)
    vgprs = [int(x) for x in re.findall(r"\.vgpr_count:\s+(\d+)", asm)]
    assert len(names) == len(vgprs) == N_INSTANCES
    for name, v in zip(names, vgprs):
        assert v <= 256, (name, v)
        if "ILi64ELi64E" in name and "ELi4EEEv" in name:
            assert v <= 168, (name, v)
