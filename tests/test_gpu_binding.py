"""The Python binding's own checks on device tensors: every malformed call
raises before anything reaches the C library, and the stream and output
arguments are honoured."""
from __future__ import annotations

import numpy as np
import pytest

import seeded_inputs as si
from tests.gpu_util import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qa():
    import torch
    import paper_2506_12355_amd as qa
    assert torch.cuda.is_available()
    qa.load_library()
    return qa


@pytest.fixture(scope="module")
def qkv():
    return [to_device(x, "bf16") for x in si.make_qkv(1, 4, 70, 64, "bf16", seed=140)]


def test_malformed_16bit_calls_raise(qa, qkv):
    import torch
    q, k, v = qkv
    with pytest.raises(ValueError):
        qa.fwd(q[0], k, v)                                   # not 4-D
    with pytest.raises(ValueError):
        qa.fwd(q, k[:, :, :60].contiguous(), v)              # k length differs
    with pytest.raises(TypeError):
        qa.fwd(q, k.half(), v)                               # mixed dtypes
    with pytest.raises(TypeError):
        qa.fwd(q.float(), k.float(), v.float())              # fp32 inputs
    with pytest.raises(ValueError):
        qa.fwd(q.transpose(2, 3), k, v)                      # q's N and d swapped
    strided = q.transpose(2, 3).contiguous().transpose(2, 3)  # q's shape, not contiguous
    assert strided.shape == q.shape and not strided.is_contiguous()
    with pytest.raises(ValueError):
        qa.fwd(strided, k, v)
    with pytest.raises(ValueError):
        qa.fwd(q, k, v, layout="nhd")
    with pytest.raises(ValueError):
        qa.fwd(q, k, v, out=torch.empty_like(q, dtype=torch.float16))
    with pytest.raises(ValueError):
        qa.fwd(q, k, v, lse=torch.empty((1, 4, 71), dtype=torch.float32, device="cuda"))
    with pytest.raises(ValueError):
        qa.fwd(q, k.cpu(), v)                                # host tensor
    # outputs on the host: rejected before the library is called (the kernel
    # would write through a host address)
    with pytest.raises(ValueError, match="out must be on"):
        qa.fwd(q, k, v, out=torch.empty(tuple(q.shape), dtype=q.dtype))
    with pytest.raises(ValueError, match="lse must be on"):
        qa.fwd(q, k, v, lse=torch.empty((1, 4, 70), dtype=torch.float32))
    # value width 32 with key width 64 is no supported pair: the library says so
    with pytest.raises(qa.QmAttnError) as e:
        qa.fwd(q, k, v[:, :, :, :32].contiguous())
    assert e.value.status == qa.QM_ERR_HEADDIM
    # three key/value heads do not divide four query heads
    k3, v3 = (x[:, :3].contiguous() for x in (k, v))
    with pytest.raises(qa.QmAttnError) as e:
        qa.fwd(q, k3, v3)
    assert e.value.status == qa.QM_ERR_SHAPE


def test_malformed_fp8_calls_raise(qa):
    import torch
    q8, k8, v8 = (torch.from_numpy(x).cuda() for x in si.make_qkv_fp8_dyadic(1, 2, 40, 128, seed=141))
    s = (1.0, 1.0, 1.0)
    with pytest.raises(TypeError):
        qa.fwd_fp8(q8.to(torch.int16), k8, v8, s)
    with pytest.raises(ValueError):
        qa.fwd_fp8(q8, k8[:, :, :30].contiguous(), v8, s)
    with pytest.raises(ValueError):
        qa.fwd_fp8(q8, k8, v8, s, layout="bhn")
    with pytest.raises(ValueError):
        qa.fwd_fp8(q8, k8, v8, s, out=torch.empty((1, 2, 40, 128), dtype=torch.float16,
                                                  device="cuda"))
    with pytest.raises(ValueError, match="out must be on"):    # host output
        qa.fwd_fp8(q8, k8, v8, s, out=torch.empty((1, 2, 40, 128), dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="lse must be on"):    # host lse
        qa.fwd_fp8(q8, k8, v8, s, lse=torch.empty((1, 2, 40), dtype=torch.float32))
    with pytest.raises(qa.QmAttnError) as e:       # FP8 runs at d = 128 only
        qa.fwd_fp8(q8[..., :64].contiguous(), k8[..., :64].contiguous(),
                   v8[..., :64].contiguous(), s)
    assert e.value.status == qa.QM_ERR_HEADDIM
    with pytest.raises(qa.QmAttnError) as e:
        qa.fwd_fp8(q8, k8, v8, (float("nan"), 1.0, 1.0))
    assert e.value.status == qa.QM_ERR_SCALE


def test_outputs_and_stream_are_honoured(qa, qkv):
    """out= and lse= are written in place and returned; a call on a side
    stream matches the call on the current stream byte for byte."""
    import torch
    q, k, v = qkv
    ref_o, ref_l = qa.fwd(q, k, v, causal=True)
    torch.cuda.synchronize()
    o = torch.full_like(q, float("nan"))
    lse = torch.full((1, 4, 70), float("nan"), device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    ro, rl = qa.fwd(q, k, v, causal=True, out=o, lse=lse, stream=s)
    s.synchronize()
    assert ro is o and rl is lse
    assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), ref_l.view(torch.int32))
    assert np.isfinite(lse.cpu().numpy()).all()
