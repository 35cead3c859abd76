"""Pins of the decode-layer oracle (oracle.af_decode_layer_steps): closed forms
for sequences whose only cached token is the appended one, where attention
returns that token's value exactly, so every other step of the layer can be
written out by hand."""
import numpy as np
import torch

import oracle
from paper_2608_01891_amd import synth

B, HQ, HKV, D, E, I = 6, 4, 2, 16, 4, 32
H = HQ * D


def _setup(ctx, residual=True, zero_experts=True, seed=31):
    a = synth.custom_attention(seed, B, HQ, HKV, D, ctx, ctx_hi=64)
    _, w, _ = synth.custom_ffn(seed, B, H, I, E=E)
    if zero_experts:
        w.w_down = torch.zeros_like(w.w_down)
    layer = synth.make_layer(seed, B, HQ, HKV, D, H, E, residual=residual)
    perm = torch.from_numpy(np.random.default_rng(seed).permutation(H))
    w_o = torch.zeros(H, H, dtype=torch.bfloat16)
    w_o[torch.arange(H), perm] = 1.0          # h[:, i] = a[:, perm[i]]
    layer.w_o = w_o
    return a, w, layer, perm


def _appended_values(layer):
    """Attention output of a sequence whose only token is the appended one:
    head h returns v_new of its kv head g = h // (HQ // HKV)."""
    g = torch.arange(HQ) // (HQ // HKV)
    return layer.v_new.to(torch.float64)[:, g, :].reshape(B, H)


def test_append_projection_residual_closed_form():
    a, w, layer, perm = _setup([1] * B)
    y, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [B])
    want = _appended_values(layer)[:, perm] + layer.x_in.to(torch.float64)
    assert torch.equal(y, want)


def test_without_layer_input():
    a, w, layer, perm = _setup([1] * B, residual=False)
    y, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [2, 4])
    assert torch.equal(y, _appended_values(layer)[:, perm])


def test_second_step_feeds_y_back_as_input():
    """Step 2 attends over the same single token (q does not matter) and adds
    step 1's output as the layer input: y2 = 2 perm(v) + x."""
    a, w, layer, perm = _setup([1] * B)
    y2, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [3, 3], L=2)
    want = 2 * _appended_values(layer)[:, perm] + layer.x_in.to(torch.float64)
    assert torch.equal(y2, want)


def test_moe_block_on_the_projected_state():
    a, w, layer, perm = _setup([1] * B, zero_experts=False)
    y, logits = oracle.af_decode_layer_steps(a, w, layer, 2, [B])
    h = _appended_values(layer)[:, perm] + layer.x_in.to(torch.float64)
    ref, ref_lg, _ = oracle.moe_block(h, layer.norm_weight, layer.eps, layer.router_weight, w.w_gate,
                                      w.w_up, w.w_down, 2, True)
    assert torch.allclose(y, ref, rtol=1e-13, atol=1e-13)
    assert torch.allclose(logits[0], ref_lg, rtol=1e-13, atol=1e-13)


def test_older_tokens_and_microbatch_split_invariance():
    """With longer contexts the appended token is the last of several; the
    result does not depend on how the batch is cut into microbatches, and the
    cache the attention read holds the new token at position ctx - 1."""
    ctx = [1, 17, 40, 5, 33, 64]
    a, w, layer, _ = _setup(ctx, zero_experts=False)
    y1, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [B], L=2)
    y3, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [1, 2, 3], L=2)
    assert torch.allclose(y1, y3, rtol=1e-13, atol=1e-13)
    kc, vc = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, layer.k_new,
                              layer.v_new)
    att = oracle.attention_decode(a.q, kc, vc, a.block_table, a.context_lens)
    h = att.reshape(B, H) @ layer.w_o.to(torch.float64).T + layer.x_in.to(torch.float64)
    one, _ = oracle.af_decode_layer_steps(a, w, layer, 2, [B], L=1)
    ref, _, _ = oracle.moe_block(h, layer.norm_weight, layer.eps, layer.router_weight, w.w_gate, w.w_up,
                                 w.w_down, 2, True)
    assert torch.allclose(one, ref, rtol=1e-13, atol=1e-13)
