"""Pins of the causal prefill-attention oracle: a scalar brute force, torch's
scaled_dot_product_attention with its causal mask, closed forms, causality,
packing invariance, and agreement of each prompt's last row with the
(separately pinned) decode-attention oracle over a paged copy of its K/V."""
import math

import numpy as np
import torch
import torch.nn.functional as F

import oracle
from paper_2608_01891_amd import synth


def _rand(lens, Hq, Hkv, D, seed):
    rng = np.random.default_rng(seed)
    T = sum(lens)
    cu = torch.tensor([0] + list(np.cumsum(lens)), dtype=torch.int32)
    q = torch.tensor(rng.standard_normal((T, Hq, D)))
    k = torch.tensor(rng.standard_normal((T, Hkv, D)))
    v = torch.tensor(rng.standard_normal((T, Hkv, D)))
    return q, k, v, cu


def test_bruteforce_scalar_loops():
    lens = [3, 1, 5]
    Hq, Hkv, D = 4, 2, 4
    q, k, v, cu = _rand(lens, Hq, Hkv, D, 1)
    scale = 0.37
    out = oracle.attention_prefill(q, k, v, cu, scale=scale)
    ref = torch.zeros_like(out)
    for b in range(len(lens)):
        s0 = int(cu[b])
        for i in range(lens[b]):
            for h in range(Hq):
                g = h // (Hq // Hkv)
                s = [scale * sum(float(q[s0 + i, h, d]) * float(k[s0 + j, g, d]) for d in range(D))
                     for j in range(i + 1)]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                for d in range(D):
                    ref[s0 + i, h, d] = sum(e[j] * float(v[s0 + j, g, d]) for j in range(i + 1)) / sum(e)
    assert torch.allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_matches_sdpa_causal():
    lens = [17, 40, 1, 33]
    Hq, Hkv, D = 8, 2, 16
    q, k, v, cu = _rand(lens, Hq, Hkv, D, 2)
    out = oracle.attention_prefill(q, k, v, cu)
    G = Hq // Hkv
    for b in range(len(lens)):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        qb = q[s0:s1].permute(1, 0, 2)                          # [Hq, n, D]
        kb = k[s0:s1].permute(1, 0, 2).repeat_interleave(G, 0)  # [Hq, n, D]
        vb = v[s0:s1].permute(1, 0, 2).repeat_interleave(G, 0)
        ref = F.scaled_dot_product_attention(qb, kb, vb, is_causal=True)
        assert torch.allclose(out[s0:s1].permute(1, 0, 2), ref, rtol=1e-10, atol=1e-12)


def test_single_token_prompts_return_v():
    lens = [1, 1, 1]
    q, k, v, cu = _rand(lens, 4, 1, 8, 3)
    out = oracle.attention_prefill(q, k, v, cu)
    assert torch.equal(out, v.expand(3, 4, 8))


def test_identical_keys_give_prefix_means():
    lens = [9, 20]
    Hq, Hkv, D = 2, 1, 8
    q, k, v, cu = _rand(lens, Hq, Hkv, D, 4)
    k[:] = k[0]
    out = oracle.attention_prefill(q, k, v, cu)
    for b in range(2):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        csum = torch.cumsum(v[s0:s1, 0], dim=0)
        mean = csum / torch.arange(1, s1 - s0 + 1, dtype=torch.float64)[:, None]
        for h in range(Hq):
            assert torch.allclose(out[s0:s1, h], mean, rtol=1e-12, atol=1e-13)


def test_causal_future_tokens_do_not_matter():
    lens = [24]
    q, k, v, cu = _rand(lens, 4, 2, 8, 5)
    out = oracle.attention_prefill(q, k, v, cu)
    k2, v2 = k.clone(), v.clone()
    k2[11:] = 1e3
    v2[11:] = float("nan")
    out2 = oracle.attention_prefill(q, k2, v2, cu)
    assert torch.equal(out[:11], out2[:11])
    assert not torch.equal(out[11:], out2[11:])


def test_packing_invariance_and_empty_prompts():
    lens = [0, 13, 0, 7, 0]
    q, k, v, cu = _rand(lens, 4, 2, 8, 6)
    out = oracle.attention_prefill(q, k, v, cu)
    one = oracle.attention_prefill(q[:13], k[:13], v[:13], torch.tensor([0, 13], dtype=torch.int32))
    two = oracle.attention_prefill(q[13:], k[13:], v[13:], torch.tensor([0, 7], dtype=torch.int32))
    assert torch.equal(out, torch.cat([one, two]))
    rows = [0, 12, 19]
    part = oracle.attention_prefill(q, k, v, cu, rows=rows)
    assert torch.equal(part[rows], out[rows])
    assert torch.count_nonzero(part[[1, 5, 13]]) == 0


def test_last_row_equals_decode_over_paged_copy():
    """The last prompt token attends to the whole prompt, which is the decode
    oracle's definition with ctx = prompt length over a paged cache."""
    lens = [37, 16, 1]
    Hq, Hkv, D, bs = 8, 2, 16, 16
    q, k, v, cu = _rand(lens, Hq, Hkv, D, 7)
    out = oracle.attention_prefill(q, k, v, cu)
    rng = np.random.default_rng(8)
    nblk = [-(-n // bs) for n in lens]
    perm = rng.permutation(sum(nblk))
    kc = torch.full((sum(nblk), Hkv, bs, D), float("nan"), dtype=torch.float64)
    vc = torch.full((sum(nblk), Hkv, D, bs), float("nan"), dtype=torch.float64)
    table = torch.full((len(lens), max(nblk)), -1, dtype=torch.int32)
    pos = 0
    for b, n in enumerate(lens):
        for j in range(nblk[b]):
            p = int(perm[pos]); pos += 1
            table[b, j] = p
            for o in range(bs):
                t = j * bs + o
                if t < n:
                    kc[p, :, o, :] = k[int(cu[b]) + t]
                    vc[p, :, :, o] = v[int(cu[b]) + t]
    last = (cu[1:] - 1).long()
    dec = oracle.attention_decode(q[last], kc, vc, table, torch.tensor(lens, dtype=torch.int32))
    assert torch.allclose(dec, out[last], rtol=1e-12, atol=1e-13)


def test_generator_shapes():
    w = synth.make_prefill(9, [5, 0, 3], 4, 2, 128)
    assert w.q.shape == (8, 4, 128) and w.k.shape == (8, 2, 128) and w.v.dtype == torch.bfloat16
    assert w.cu_seqlens.tolist() == [0, 5, 5, 8] and w.T == 8 and w.max_seqlen == 5
    assert not torch.equal(w.q[:, :2].float(), w.k.float())
