"""The gfx950 kernels as compiled (CPU only: hipcc cross-compiles the device code).

* every direct HBM -> LDS load is clear of the VALU-write-SGPR hazard on
  every path into it (its inline assembly carries only the one wait state
  the M0 write needs);
* no packed fp32 instruction appears in device code;
* no kernel spills VGPRs or uses scratch memory.
"""
from __future__ import annotations

import os
import re
import subprocess

import pytest

from paper_2506_12355_amd import build as qbuild
from tests.asm_hazards import dma_sgpr_hazards, dma_sgpr_hazards_cfg, instructions, is_direct_load


def _compile(tmp_path_factory, extra):
    try:
        cc = qbuild.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "attn.s")
    flags = [f for f in qbuild.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    cmd = ([cc] + flags + extra + ["--cuda-device-only", "-S", "-I", qbuild.INCLUDE, "-I", qbuild.CSRC,
                                   "-o", out, os.path.join(qbuild.CSRC, "attn_fwd_gfx950.hip")])
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return open(out).read()


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    return _compile(tmp_path_factory, [])


@pytest.fixture(scope="module")
def asm_debug(tmp_path_factory):
    """The checking build (a barrier after every key block)."""
    return _compile(tmp_path_factory, ["-DQM_DEBUG_SYNC"])


def _kernel_texts(text):
    """name -> assembly text of the kernel's body, one per kernel instance."""
    out = {}
    for m in re.finditer(r"^(_Z\w*attn_fwd_kernel\w*):\s*(?:;.*)?$", text, flags=re.M):
        end = text.index(".Lfunc_end", m.end())   # a kernel may hold several s_endpgm
        out[m.group(1)] = text[m.end():end]
    return out


def _kernels(text):
    """name -> instruction list, one per kernel instance."""
    return {name: instructions(body) for name, body in _kernel_texts(text).items()}


N_INSTANCES = 24   # eight waves: 16-bit (64,64), (128,128), (192,128) x dtype x mask and FP8
                   # (128,128) x mask; four waves: the same without (192,128)


def test_all_instances_compiled(asm):
    names = list(_kernels(asm))
    assert len(names) == N_INSTANCES
    assert sum("ELi8EEEv" in n for n in names) == 14
    assert sum("ELi4EEEv" in n for n in names) == 10


def _check_direct_loads(text):
    kernels = _kernel_texts(text)
    assert len(kernels) == N_INSTANCES
    for name, body in kernels.items():
        insts = instructions(body)
        assert any(is_direct_load(i) for i in insts), name
        bad = dma_sgpr_hazards_cfg(body)
        assert not bad, f"{name}: {bad[:3]}"
        # each direct load comes right after its own s_nop: the wait state
        # that separates it from the write of M0 (its LDS address)
        for i, inst in enumerate(insts):
            if is_direct_load(inst):
                assert i > 0 and insts[i - 1].startswith("s_nop"), (name, i, inst)


def test_direct_loads_have_no_sgpr_hazard(asm):
    _check_direct_loads(asm)


def test_direct_loads_have_no_sgpr_hazard_in_the_checking_build(asm_debug):
    _check_direct_loads(asm_debug)


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


LOAD = "buffer_load_dwordx4 v1, s[4:7], 0 offen lds"


def test_path_aware_checker_sees_planted_hazards():
    """The scan over every path into a load: a writer before a branch to the
    load's block, on the fall-through edge, at the end of a loop whose first
    block holds the load, of M0, and of a carry destination, are all reported;
    a writer whose block cannot fall through, or five wait states away, is not."""
    across_branch = f"""
      v_readlane_b32 s5, v243, 3
      s_cbranch_scc1 .LBB0_9
      s_mov_b32 s0, 0
      s_mov_b32 s1, 0
      s_mov_b32 s2, 0
      s_mov_b32 s3, 0
      s_mov_b32 s8, 0
      s_branch .LBB0_10
    .LBB0_9:
      s_nop 0
      {LOAD}
    .LBB0_10:
      s_endpgm
    """
    assert len(dma_sgpr_hazards_cfg(across_branch)) == 1
    fall_through = f"""
      v_readfirstlane_b32 s6, v1
    .LBB0_3:
      s_nop 0
      {LOAD}
    """
    assert len(dma_sgpr_hazards_cfg(fall_through)) == 1
    no_fall_through = f"""
      v_readfirstlane_b32 s6, v1
      s_branch .LBB0_5
    .LBB0_3:
      s_nop 0
      {LOAD}
    .LBB0_5:
      s_endpgm
    """
    assert dma_sgpr_hazards_cfg(no_fall_through) == []
    back_edge = f"""
    .LBB0_2:
      s_nop 0
      {LOAD}
      s_nop 2
      v_cmp_gt_i32_e64 s[4:5], v1, v2
      s_cbranch_scc1 .LBB0_2
      s_endpgm
    """
    assert len(dma_sgpr_hazards_cfg(back_edge)) == 1
    m0 = f"""
      v_readfirstlane_b32 m0, v1
      s_nop 1
      {LOAD}
    """
    assert len(dma_sgpr_hazards_cfg(m0)) == 1
    carry = f"""
      v_add_co_u32_e64 v2, s[6:7], v3, v4
      {LOAD}
    """
    assert len(dma_sgpr_hazards_cfg(carry)) == 1
    far = f"""
      v_readlane_b32 s5, v243, 3
      s_nop 3
      s_nop 0
      {LOAD}
    """
    assert dma_sgpr_hazards_cfg(far) == []


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
