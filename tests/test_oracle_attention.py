"""Pins of the attention oracle: closed forms, invariants, brute force on an
unpaged layout, and torch's scaled_dot_product_attention as an independent
library routine."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2608_01891_amd import synth


def _page(kd, vd, ctx, rng, bs=16):
    """Pack dense per-sequence K/V [Hkv, ctx_b, D] into the paged pools (test's own paging)."""
    Hkv, D = kd[0].shape[0], kd[0].shape[2]
    nblk = [-(-c // bs) for c in ctx]
    N = sum(nblk)
    perm = rng.permutation(N)
    kc = torch.full((N, Hkv, bs, D), float("nan"), dtype=torch.float64)
    vc = torch.full((N, Hkv, D, bs), float("nan"), dtype=torch.float64)
    table = torch.full((len(ctx), max(nblk)), -1, dtype=torch.int32)
    pos = 0
    for b, c in enumerate(ctx):
        for j in range(nblk[b]):
            p = int(perm[pos]); pos += 1
            table[b, j] = p
            for o in range(bs):
                t = j * bs + o
                if t < c:
                    kc[p, :, o, :] = kd[b][:, t, :]
                    vc[p, :, :, o] = vd[b][:, t, :]
    return kc, vc, table


def _brute(q, kd, vd, ctx, scale):
    """Scalar-loop attention on the dense (unpaged) arrays."""
    B, Hq, D = q.shape
    Hkv = kd[0].shape[0]
    out = torch.zeros(B, Hq, D, dtype=torch.float64)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            s = [scale * sum(float(q[b, h, d]) * float(kd[b][g, t, d]) for d in range(D))
                 for t in range(ctx[b])]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for d in range(D):
                out[b, h, d] = sum(e[t] * float(vd[b][g, t, d]) for t in range(ctx[b])) / z
    return out


def test_bruteforce_unpaged_tiny():
    rng = np.random.default_rng(3)
    ctx = [1, 17, 33, 16]
    B, Hq, Hkv, D = 4, 4, 2, 8
    q = torch.tensor(rng.standard_normal((B, Hq, D)))
    kd = [torch.tensor(rng.standard_normal((Hkv, c, D))) for c in ctx]
    vd = [torch.tensor(rng.standard_normal((Hkv, c, D))) for c in ctx]
    kc, vc, table = _page(kd, vd, ctx, rng)
    cl = torch.tensor(ctx, dtype=torch.int32)
    got = oracle.attention_decode(q, kc, vc, table, cl)
    ref = _brute(q, kd, vd, ctx, 1 / math.sqrt(D))
    assert torch.allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_matches_sdpa_gqa_on_tiny_layer():
    w = synth.tiny_layer().attn
    got = oracle.attention_decode(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens)
    for b in range(w.B):
        c = int(w.context_lens[b])
        k, v = oracle.gather_sequence(w.k_cache, w.v_cache, w.block_table, b, c)
        # gather with the test's own indexing, independent of the oracle's helper
        phys = [int(w.block_table[b, j // 16]) for j in range(c)]
        k2 = torch.stack([w.k_cache[phys[j], :, j % 16, :] for j in range(c)], 1).double()
        v2 = torch.stack([w.v_cache[phys[j], :, :, j % 16] for j in range(c)], 1).double()
        assert torch.equal(k, k2) and torch.equal(v, v2)
        ref = F.scaled_dot_product_attention(w.q[b].double()[None, :, None, :], k2[None],
                                             v2[None], enable_gqa=True)[0, :, 0, :]
        assert torch.allclose(got[b], ref, rtol=1e-12, atol=1e-12)


def test_context_one_returns_v():
    a = synth.custom_attention(5, 3, 8, 2, 64, [1, 1, 1])
    got = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    for b in range(3):
        p = int(a.block_table[b, 0])
        for h in range(8):
            assert torch.equal(got[b, h], a.v_cache[p, h // 4, :, 0].double())


def test_identical_keys_give_mean_of_v():
    a = synth.custom_attention(6, 2, 4, 1, 64, [37, 50])
    k = a.k_cache.clone()
    k[:] = k[0, 0, 0]
    got = oracle.attention_decode(a.q, k, a.v_cache, a.block_table, a.context_lens)
    for b in range(2):
        _, v = oracle.gather_sequence(k, a.v_cache, a.block_table, b, int(a.context_lens[b]))
        assert torch.allclose(got[b], v[0].mean(0).expand(4, -1), rtol=1e-12, atol=1e-14)


def test_weights_sum_to_one_and_positive():
    a = synth.tiny_layer().attn
    for b in range(a.B):
        p = oracle.attention_weights(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens, b)
        assert p.shape == (a.Hq, int(a.context_lens[b]))
        assert (p > 0).all()
        assert torch.allclose(p.sum(1), torch.ones(a.Hq, dtype=torch.float64), atol=1e-14)


def test_block_permutation_invariance():
    a = synth.tiny_layer().attn
    ref = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    perm = torch.from_numpy(np.random.default_rng(9).permutation(a.num_blocks))
    inv = torch.empty_like(perm); inv[perm] = torch.arange(a.num_blocks)
    table = a.block_table.clone()
    valid = table >= 0
    table[valid] = inv[table[valid].long()].int()
    got = oracle.attention_decode(a.q, a.k_cache[perm], a.v_cache[perm], table, a.context_lens)
    assert torch.equal(got, ref)


def test_tail_slots_are_ignored():
    a = synth.tiny_layer().attn
    ref = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    k = a.k_cache.clone().float(); v = a.v_cache.clone().float()
    for b, c in enumerate(a.context_lens.tolist()):
        last = int(a.block_table[b, (c - 1) // 16])
        k[last, :, c % 16 or 16:, :] = float("nan")
        v[last, :, :, c % 16 or 16:] = float("nan")
    got = oracle.attention_decode(a.q, k, v, a.block_table, a.context_lens)
    assert torch.equal(got, ref)


def test_scaling_v_scales_output_and_mha_special_case():
    a = synth.custom_attention(7, 2, 4, 4, 64, [40, 9])
    ref = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    got = oracle.attention_decode(a.q, a.k_cache, a.v_cache.double() * 2, a.block_table,
                                  a.context_lens)
    assert torch.equal(got, 2 * ref)
    for b in range(2):
        k, v = oracle.gather_sequence(a.k_cache, a.v_cache, a.block_table, b,
                                      int(a.context_lens[b]))
        sd = F.scaled_dot_product_attention(a.q[b].double()[:, None, :], k, v)[:, 0, :]
        assert torch.allclose(ref[b], sd, rtol=1e-12, atol=1e-12)


def test_dominant_score_selects_its_value():
    a = synth.custom_attention(8, 1, 2, 1, 64, [30])
    q = torch.zeros(1, 2, 64, dtype=torch.float64); q[0, :, 0] = 1.0
    k = a.k_cache.double().clone(); k[..., 0] = 0.0
    p = int(a.block_table[0, 1]); k[p, 0, 3, 0] = 400.0      # token 19, score 50
    got = oracle.attention_decode(q, k, a.v_cache, a.block_table, a.context_lens)
    assert torch.allclose(got[0, 0], a.v_cache[p, 0, :, 3].double(), atol=1e-18)


def test_closed_form_two_tokens():
    # D = 4 (scale 1/2); scores 1 and 0; weights sigmoid(1) and 1 - sigmoid(1)
    kc = torch.zeros(1, 1, 16, 4, dtype=torch.float64); kc[0, 0, 0, 0] = 2.0
    vc = torch.zeros(1, 1, 4, 16, dtype=torch.float64); vc[0, 0, 0, 0] = 1.0; vc[0, 0, 1, 1] = 1.0
    q = torch.tensor([[[1.0, 0, 0, 0]]], dtype=torch.float64)
    got = oracle.attention_decode(q, kc, vc, torch.tensor([[0]], dtype=torch.int32),
                                  torch.tensor([2], dtype=torch.int32))
    s = 1.0 / (1.0 + math.exp(-1.0))
    assert torch.allclose(got[0, 0], torch.tensor([s, 1 - s, 0, 0], dtype=torch.float64),
                          rtol=0, atol=1e-15)


def test_empty_context_gives_zero():
    a = synth.custom_attention(9, 2, 4, 2, 64, [0, 5], ctx_hi=16)
    got = oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens)
    assert torch.equal(got[0], torch.zeros(4, 64, dtype=torch.float64))
    assert got[1].abs().sum() > 0
