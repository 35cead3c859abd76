"""Seeded random shape sweep of every operator against the oracle: sizes drawn
from a fixed generator (not hand-picked) within each entry point's supported
range, small enough for the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
RNG_SEED = 20260801


def _cases(n, draw, stream):
    """n shapes from draw(rng); each case carries its own input seed."""
    rng = np.random.default_rng([RNG_SEED, stream])
    return [(1000 * stream + i,) + draw(rng) for i in range(n)]


def _attn_case(rng):
    D = int(rng.choice([64, 128]))
    Hkv = int(rng.integers(1, 5))
    G = int(rng.choice([1, 2, 4, 8, 16]))
    B = int(rng.integers(1, 9))
    ctx = [int(c) for c in rng.integers(0, 700, B)]
    split = int(rng.choice([0, 128, 256, 512]))
    return D, Hkv * G, Hkv, ctx, split


@pytest.mark.parametrize("case", _cases(24, _attn_case, 1))
def test_decode_attention_sweep(gpu_lib, case):
    seed, D, Hq, Hkv, ctx, split = case
    a = synth.custom_attention(seed, len(ctx), Hq, Hkv, D, ctx, ctx_hi=max(max(ctx), 1) + 30)
    out = aflex.attn_decode(a.to(DEV), split_tokens=split).cpu()
    ref = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    check_rows(out, ref, what=f"attention sweep {case}")


def _ffn_case(rng):
    T = int(rng.integers(1, 300))
    H = 64 * int(rng.integers(1, 9))
    I = 64 * int(rng.integers(1, 12))
    return T, H, I


@pytest.mark.parametrize("case", _cases(20, _ffn_case, 2))
def test_swiglu_sweep(gpu_lib, case):
    seed, T, H, I = case
    x, w, _ = synth.custom_ffn(seed, T, H, I)
    y = aflex.ffn_swiglu(x.to(DEV), w.to(DEV)).cpu()
    check_rows(y, oracle.swiglu_ffn(x, w.w_gate, w.w_up, w.w_down), what=f"swiglu sweep {case}")


def _moe_case(rng):
    E = int(rng.choice([1, 2, 3, 8, 16, 64]))
    k = int(rng.integers(1, min(E, 8) + 1))
    T = int(rng.integers(1, 400))
    H = 64 * int(rng.integers(1, 5))
    I = 64 * int(rng.integers(1, 5))
    return T, H, I, E, k


@pytest.mark.parametrize("case", _cases(20, _moe_case, 3))
def test_moe_sweep(gpu_lib, case):
    seed, T, H, I, E, k = case
    x, w, logits = synth.custom_ffn(seed, T, H, I, E=E)
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    ids, _ = oracle.route_topk(logits, k)
    assert torch.equal(r["topk_ids"].cpu().long(), ids)
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k)
    check_rows(y.cpu(), ref, what=f"moe sweep {case}")


def _prefill_case(rng):
    Hkv = int(rng.integers(1, 4))
    G = int(rng.choice([1, 2, 4, 8]))
    lens = [int(n) for n in rng.integers(0, 300, int(rng.integers(1, 5)))]
    return Hkv * G, Hkv, lens


@pytest.mark.parametrize("case", _cases(16, _prefill_case, 4))
def test_prefill_sweep(gpu_lib, case):
    seed, Hq, Hkv, lens = case
    if sum(lens) == 0:
        lens = lens + [1]
    p = synth.make_prefill(seed, lens, Hq, Hkv, 128)
    out = aflex.attn_prefill(p.to(DEV)).cpu()
    ref = oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens)
    check_rows(out, ref, what=f"prefill sweep {case}")


def _long_prefill_case(rng):
    """A batch holding one prompt of 2048-2600 tokens (so both prefill kernel
    shapes are drawn: two query heads per work-group for an even number of
    heads per KV group, one head otherwise) beside 0-3 prompts of 0-2600."""
    Hkv = int(rng.integers(1, 3))
    G = int(rng.choice([1, 2, 3, 4, 8, 16]))
    lens = [int(n) for n in rng.integers(0, 2601, int(rng.integers(0, 4)))]
    pos = int(rng.integers(0, len(lens) + 1))
    lens.insert(pos, int(rng.integers(2048, 2601)))
    return Hkv * G, Hkv, lens


@pytest.mark.parametrize("case", _cases(8, _long_prefill_case, 5))
def test_long_prefill_sweep(gpu_lib, case):
    """Rows checked per prompt: first, last, both edges of the first two
    64-row blocks, the middle and three random rows."""
    seed, Hq, Hkv, lens = case
    p = synth.make_prefill(seed, lens, Hq, Hkv, 128, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    rng = np.random.default_rng(seed)
    rows, start = set(), 0
    for n in lens:
        if n:
            picks = {0, min(63, n - 1), min(64, n - 1), min(127, n - 1), min(128, n - 1), n // 2, n - 1}
            picks |= {int(r) for r in rng.integers(0, n, 3)}
            rows |= {start + r for r in picks}
        start += n
    rows = sorted(rows)
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens, rows=rows)
    check_rows(out[rows], ref[rows], what=f"long prefill sweep {case}")
