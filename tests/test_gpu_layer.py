"""The whole decode layer on the interleaved A/F step (KV append, attention,
output projection | RMSNorm, router, MoE, residual) vs the oracle, through
the C ABI.

The router logits are computed from the hidden state that crossed the A/F
boundary, which the GPU holds in bf16 and the oracle in float64, so a
routing decision is unique only where the oracle's top-k margin exceeds that
rounding: those rows are compared with the oracle; the few near ties are
left out (at most 2 or 5% of the rows)."""
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
MARGIN = 2e-2


def _margins(logits, k):
    s = torch.sort(logits.double(), dim=1, descending=True).values
    return (s[:, :k] - s[:, 1:k + 1]).min(dim=1).values


def _clear_rows(logit_steps, k):
    clear = torch.ones(logit_steps[0].shape[0], dtype=torch.bool)
    for lg in logit_steps:
        clear &= _margins(lg, k) > MARGIN
    assert int((~clear).sum()) <= max(2, clear.numel() // 20)
    return clear


def _small(seed, ctx, E=4, residual=True):
    B = len(ctx)
    a = synth.custom_attention(seed, B, 8, 2, 64, ctx, ctx_hi=max(ctx) + 16)
    _, w, _ = synth.custom_ffn(seed, B, 512, 256, E=E)
    layer = synth.make_layer(seed, B, 8, 2, 64, 512, E, residual=residual)
    return a, w, layer


@pytest.mark.parametrize("mbs,L,residual", [([8], 1, True), ([4, 4], 1, False), ([2, 2, 2, 2], 2, True),
                                            ([3, 5], 2, False), ([1, 1, 6], 3, True)])
def test_small_layer(gpu_lib, mbs, L, residual):
    ctx = [5, 17, 40, 1, 33, 300, 9, 64]
    a, w, layer = _small(90, ctx, residual=residual)
    ad = a.to(DEV)
    y = aflex.af_layer_step(ad, w.to(DEV), layer.to(DEV), 2, mbs, L=L).cpu()
    ref, logits = oracle.af_decode_layer_steps(a, w, layer, 2, mbs, L=L)
    clear = _clear_rows(logits, 2)
    check_rows(y[clear], ref[clear], what=f"decode layer mbs={mbs} L={L}")
    # the append wrote the new token at position ctx - 1 of each sequence, bit-exact
    rk, rv = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, layer.k_new, layer.v_new)
    assert torch.equal(ad.k_cache.cpu(), rk) and torch.equal(ad.v_cache.cpu(), rv)


def test_repeated_steps_are_deterministic(gpu_lib):
    a, w, layer = _small(91, [3, 70, 200, 1, 16, 47, 129, 9])
    ad, wd, ld = a.to(DEV), w.to(DEV), layer.to(DEV)
    ys = [aflex.af_layer_step(ad, wd, ld, 2, [3, 5]).clone() for _ in range(3)]
    torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1]) and torch.equal(ys[1], ys[2])


def test_mixtral_layer_all_rows(gpu_lib):
    """The pipeline workload (B = 256, 32/8 heads, long contexts, top-2 of 8
    Mixtral experts, M = 4 microbatches of 64) as a whole decode layer:
    every row against the oracle."""
    wl = synth.af_pipeline(device=DEV)
    a, f = wl.attn, wl.ffn
    layer = synth.make_layer(40, a.B, a.Hq, a.Hkv, a.D, f.H, f.E, device=DEV)
    a_cpu = a.to("cpu")  # the pools before the append
    y = aflex.af_layer_step(a, f, layer, 2, wl.microbatches).cpu()
    ref, logits = oracle.af_decode_layer_steps(a_cpu, f.to("cpu"), layer.to("cpu"), 2, [a.B])
    clear = _clear_rows(logits, 2)
    check_rows(y[clear], ref[clear], what="Mixtral decode layer M=4 (all clear rows)")
