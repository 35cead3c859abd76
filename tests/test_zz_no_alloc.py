"""The no-allocation decode attention (static device scratch) against the
workspace entry point, through the C ABI: bitwise the same output on two
calls in a row, the second with a smaller input, and at the Qwen3-32B
workload's full size."""
import pytest
import torch

from paper_2608_01891_amd import aflex, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _pair(a, **kw):
    ref = aflex.attn_decode(a, **kw)
    out = torch.full_like(ref, float("nan"))
    aflex.attn_decode_noalloc(a, out, **kw)
    torch.cuda.synchronize()
    return ref, out


def test_two_calls_second_smaller(gpu_lib):
    big = synth.custom_attention(61, 12, 32, 4, 128, [1, 700, 1500, 33, 0, 2048, 17, 999, 1024, 5, 640, 1300],
                                 ctx_hi=2048).to(DEV)
    small = synth.custom_attention(62, 3, 8, 2, 64, [40, 1, 300], ctx_hi=320).to(DEV)
    r1, o1 = _pair(big, split_tokens=256)
    r2, o2 = _pair(small)
    assert torch.equal(o1, r1)
    assert torch.equal(o2, r2)
    # the first call's output is untouched by the second
    r1b, o1b = _pair(big, split_tokens=256)
    assert torch.equal(o1b, r1)


def test_qwen3_workload(gpu_lib):
    a = synth.qwen3_attention(device=DEV).attn
    ref, out = _pair(a)
    assert torch.equal(out, ref)
    small = synth.tiny_layer(device=DEV).attn
    ref2, out2 = _pair(small)
    assert torch.equal(out2, ref2)
