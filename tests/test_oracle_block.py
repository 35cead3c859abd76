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


def test_rmsnorm_bruteforce_and_invariants():
    rng = np.random.default_rng(94)
    x = torch.from_numpy(rng.standard_normal((3, 6)))
    g = torch.from_numpy(rng.standard_normal(6))
    y = oracle.rmsnorm(x, g, 1e-5)
    for t in range(3):
        ms = sum(float(v) ** 2 for v in x[t]) / 6
        for i in range(6):
            assert abs(float(y[t, i]) - float(x[t, i]) / math.sqrt(ms + 1e-5) * float(g[i])) < 1e-12
    # scale invariance without eps; a constant row maps to gamma (unit gain) times its sign
    assert torch.allclose(oracle.rmsnorm(5.0 * x, g, 0.0), oracle.rmsnorm(x, g, 0.0), rtol=1e-13)
    c = torch.full((1, 6), -3.0, dtype=torch.float64)
    assert torch.allclose(oracle.rmsnorm(c, torch.ones(6, dtype=torch.float64), 0.0),
                          -torch.ones(1, 6, dtype=torch.float64))


def test_moe_block_routes_on_normalised_coordinates_and_adds_residual():
    # one-hot router rows: logit e is coordinate e of the normalised input
    x, w, _ = synth.custom_ffn(95, 5, 64, 64, E=4)
    gamma = torch.ones(64, dtype=torch.bfloat16)
    wr = torch.zeros(4, 64, dtype=torch.float64)
    for e in range(4):
        wr[e, e] = 1.0
    y, logits, ids = oracle.moe_block(x, gamma, 1e-6, wr, w.w_gate, w.w_up, w.w_down, 2, False)
    xn = oracle.rmsnorm(x, gamma, 1e-6)
    assert torch.equal(logits, xn[:, :4])
    ref_ids = np.argsort(-xn[:, :4].numpy(), axis=1, kind="stable")[:, :2]
    assert np.array_equal(ids.numpy(), ref_ids)
    y2, _, _ = oracle.moe_block(x, gamma, 1e-6, wr, w.w_gate, w.w_up, w.w_down, 2, True)
    assert torch.allclose(y2 - y, x.double(), rtol=0, atol=1e-15)
    ref, _, _ = oracle.moe_ffn(xn, xn[:, :4], w.w_gate, w.w_up, w.w_down, 2)
    assert torch.equal(y, ref)


def test_kv_write_one_token_each_is_kv_append():
    a = synth.custom_attention(94, 4, 8, 2, 64, [1, 16, 17, 40], ctx_hi=48)
    kn = torch.randn(4, 2, 64).to(torch.bfloat16)
    vn = torch.randn(4, 2, 64).to(torch.bfloat16)
    cu = torch.arange(5, dtype=torch.int32)
    k1, v1 = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, vn)
    k2, v2 = oracle.kv_write(a.k_cache, a.v_cache, a.block_table, a.context_lens, cu, kn, vn)
    assert torch.equal(k1, k2) and torch.equal(v1, v2)


def test_kv_write_prefill_roundtrip_and_chunk_preserves_prefix():
    ctx = [33, 16, 7, 0]
    a = synth.custom_attention(95, 4, 4, 2, 16, ctx, ctx_hi=48)
    new = [33, 16, 3, 0]                 # prompts, a full-block prompt, a 3-token chunk, nothing
    cu = torch.tensor([0] + list(np.cumsum(new)), dtype=torch.int32)
    T = int(cu[-1])
    kn = torch.randn(T, 2, 16).to(torch.bfloat16)
    vn = torch.randn(T, 2, 16).to(torch.bfloat16)
    k, v = oracle.kv_write(a.k_cache, a.v_cache, a.block_table, a.context_lens, cu, kn, vn)
    for b, (c, n) in enumerate(zip(ctx, new)):
        kg, vg = oracle.gather_sequence(k, v, a.block_table, b, c)
        k0, v0 = oracle.gather_sequence(a.k_cache, a.v_cache, a.block_table, b, c)
        s0 = int(cu[b])
        assert torch.equal(kg[:, c - n:], kn[s0:s0 + n].permute(1, 0, 2).double())
        assert torch.equal(vg[:, c - n:], vn[s0:s0 + n].permute(1, 0, 2).double())
        assert torch.equal(kg[:, :c - n], k0[:, :c - n]) and torch.equal(vg[:, :c - n], v0[:, :c - n])
    touched = int((k != a.k_cache).any(dim=(1, 3)).sum())
    assert touched == sum(new)


def test_prefill_write_then_decode_equals_prefill_last_row():
    lens = [21, 16]
    p = synth.make_prefill(96, lens, 4, 2, 16)
    a = synth.custom_attention(96, 2, 4, 2, 16, lens, ctx_hi=32)
    k, v = oracle.kv_write(a.k_cache, a.v_cache, a.block_table, a.context_lens, p.cu_seqlens, p.k, p.v)
    last = (p.cu_seqlens[1:] - 1).long()
    dec = oracle.attention_decode(p.q[last], k, v, a.block_table, a.context_lens)
    pre = oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens)
    assert torch.allclose(dec, pre[last], rtol=1e-12, atol=1e-13)
