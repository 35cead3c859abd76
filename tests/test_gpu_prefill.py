"""HIP causal prefill attention vs the oracle (through the C ABI)."""
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.helpers import sample_rows
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _run(p, **kw):
    return aflex.attn_prefill(p.to(DEV), **kw).cpu()


@pytest.mark.parametrize("lens,Hq,Hkv", [
    ([1, 5, 0, 130, 64, 200], 8, 2),        # empty prompt, one-token prompt, ragged tails
    ([63, 64, 65, 127, 128, 129], 8, 8),    # tile edges, MHA
    ([300], 16, 1),                         # 16 query heads on one KV head
    ([257, 3], 12, 4),                      # Hq not a multiple of 8 (no head permutation)
    ([0, 0, 17], 32, 8),
])
def test_small_shapes(gpu_lib, lens, Hq, Hkv):
    p = synth.make_prefill(40 + len(lens), lens, Hq, Hkv, 128)
    out = _run(p)
    ref = oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens)
    check_rows(out, ref, what=f"prefill lens={lens} Hq={Hq} Hkv={Hkv}")


def test_one_long_prompt_full(gpu_lib):
    p = synth.make_prefill(47, [1000], 8, 2, 128)
    out = _run(p)
    check_rows(out, oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens), what="prefill n=1000")


def test_scale_argument(gpu_lib):
    p = synth.make_prefill(48, [70, 90], 8, 2, 128)
    out = _run(p, scale=0.3)
    check_rows(out, oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens, scale=0.3), what="prefill scale")


def test_single_token_prompts_return_v_bitwise(gpu_lib):
    p = synth.make_prefill(49, [1] * 9, 16, 4, 128)
    out = _run(p)
    G = 4
    assert torch.equal(out, p.v.repeat_interleave(G, dim=1))


def test_loose_max_seqlen_and_determinism(gpu_lib):
    p = synth.make_prefill(50, [100, 33], 8, 2, 128)
    a = _run(p)
    b = _run(p, max_seqlen=133)
    assert torch.equal(a, b)


@pytest.mark.parametrize("model,prompt_len,prompts", [("qwen3-32b", 4096, 2), ("mixtral-8x7b", 128, 32)])
def test_paper_prompt_lengths_sampled(gpu_lib, model, prompt_len, prompts):
    p = synth.prefill_workload(model, prompt_len, prompts, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    T = pc.T
    rows = sample_rows(T, 8, seed=prompt_len,
                       must=[0, 1, 127, 128, prompt_len - 1, T - 1, T - prompt_len])
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens, rows=rows)
    check_rows(out[rows], ref[rows], what=f"{model} prefill {prompts}x{prompt_len} (sampled)")
