"""Pins of the pipeline oracle: microbatch-split invariance and equality with
serial Attention-then-FFN."""
import torch

import oracle
from paper_2608_01891_amd import synth


def _small():
    a = synth.custom_attention(21, 8, 4, 2, 16, [5, 17, 40, 1, 33, 16, 9, 64])
    x, w, _ = synth.custom_ffn(21, 8, 64, 32, E=4)
    import numpy as np
    logits = torch.from_numpy(np.random.default_rng(21).standard_normal((8, 4), dtype=np.float32))
    return a, w, logits


def test_microbatch_split_invariance():
    a, w, logits = _small()
    one = oracle.af_layer_steps(a, w, logits, 2, [8], L=1)
    four = oracle.af_layer_steps(a, w, logits, 2, [2, 2, 2, 2], L=1)
    uneven = oracle.af_layer_steps(a, w, logits, 2, [3, 5], L=2)
    uneven1 = oracle.af_layer_steps(a, w, logits, 2, [8], L=2)
    assert torch.allclose(one, four, rtol=1e-13, atol=1e-18)
    assert torch.allclose(uneven, uneven1, rtol=1e-13, atol=1e-18)


def test_equals_serial_attention_then_moe():
    a, w, logits = _small()
    got = oracle.af_layer_steps(a, w, logits, 2, [4, 4], L=1)
    att = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    y, _, _ = oracle.moe_ffn(att.reshape(8, 64), logits, w.w_gate, w.w_up, w.w_down, 2)
    assert torch.allclose(got, y, rtol=1e-13, atol=1e-18)


def test_dense_ffn_variant():
    a = synth.custom_attention(22, 4, 4, 2, 16, [3, 20, 7, 31])
    _, w, _ = synth.custom_ffn(22, 4, 64, 48)
    got = oracle.af_layer_steps(a, w, None, 0, [1, 3], L=1)
    att = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    assert torch.allclose(got, oracle.swiglu_ffn(att.reshape(4, 64), w.w_gate, w.w_up, w.w_down),
                          rtol=1e-13, atol=1e-18)
