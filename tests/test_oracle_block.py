"""Pins of the KV-append and linear-projection oracles."""
import math

import numpy as np
import torch

import oracle
from paper_2608_01891_amd import synth


def test_append_writes_only_the_new_slot():
    a = synth.custom_attention(90, 4, 8, 2, 64, [1, 16, 17, 40], ctx_hi=48)
    kn = torch.randn(4, 2, 64).to(torch.bfloat16)
    vn = torch.randn(4, 2, 64).to(torch.bfloat16)
    k, v = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, vn)
    changed_k = (k != a.k_cache).any(dim=(1, 3))  # [N, 16] slots touched
    assert int(changed_k.sum()) == 4
    for b, c in enumerate(a.context_lens.tolist()):
        kg, vg = oracle.gather_sequence(k, v, a.block_table, b, c)
        assert torch.equal(kg[:, c - 1], kn[b].double()) and torch.equal(vg[:, c - 1], vn[b].double())
        k0, v0 = oracle.gather_sequence(a.k_cache, a.v_cache, a.block_table, b, c)
        assert torch.equal(kg[:, :c - 1], k0[:, :c - 1]) and torch.equal(vg[:, :c - 1], v0[:, :c - 1])


def test_append_then_attend_equals_dense_attention_with_the_new_token():
    rng = np.random.default_rng(91)
    ctx = [5, 16, 33]
    a = synth.custom_attention(91, 3, 4, 2, 16, ctx, ctx_hi=48)
    kn = torch.from_numpy(rng.standard_normal((3, 2, 16))).to(torch.bfloat16)
    vn = torch.from_numpy(rng.standard_normal((3, 2, 16))).to(torch.bfloat16)
    k, v = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, vn)
    got = oracle.attention_decode(a.q, k, v, a.block_table, a.context_lens)
    for b, c in enumerate(ctx):
        k0, v0 = oracle.gather_sequence(a.k_cache, a.v_cache, a.block_table, b, c)
        for h in range(4):
            g = h // 2
            keys = [k0[g, t] for t in range(c - 1)] + [kn[b, g].double()]
            vals = [v0[g, t] for t in range(c - 1)] + [vn[b, g].double()]
            s = [float(a.q[b, h].double() @ kk) / 4.0 for kk in keys]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            ref = sum(w * vv for w, vv in zip(e, vals)) / sum(e)
            assert torch.allclose(got[b, h], ref, rtol=1e-12, atol=1e-14)


def test_empty_context_appends_nothing():
    a = synth.custom_attention(92, 2, 4, 1, 64, [0, 3], ctx_hi=16)
    kn = torch.full((2, 1, 64), 37.0, dtype=torch.bfloat16)  # |generated values| <= 6
    k, v = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, kn)
    assert int((k != a.k_cache).sum()) == 64 and int((v != a.v_cache).sum()) == 64


def test_linear_bruteforce_and_identity():
    rng = np.random.default_rng(93)
    x = torch.from_numpy(rng.standard_normal((3, 5)))
    w = torch.from_numpy(rng.standard_normal((4, 5)))
    y = oracle.linear(x, w)
    for t in range(3):
        for n in range(4):
            assert abs(float(y[t, n]) - sum(float(x[t, kk]) * float(w[n, kk]) for kk in range(5))) < 1e-12
    assert torch.equal(oracle.linear(x, torch.eye(5, dtype=torch.float64)), x)
    assert y.shape == (3, 4)  # [T, out_features]: catches a transposed weight
