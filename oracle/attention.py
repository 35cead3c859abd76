"""Oracle: batched GQA decode attention over a paged KV cache (float64).

Test infrastructure only (see the package docstring).

Decode attention is the operator the paper calls memory-bound because every
step reads the whole, growing KV cache (section 1; section 2 "LLM Serving";
section 3.2 reports that its decode latency barely follows the GPU clock).
The definition used for one decode token of sequence b and query head h:

    g      = h // (Hq // Hkv)                   (contiguous GQA groups)
    k_j    = K[table[b, j // bs], g, j % bs, :]  for j < ctx_b
    v_j    = V[table[b, j // bs], g, :, j % bs]
    s_j    = scale * <q[b, h], k_j>,  scale = 1/sqrt(D) unless given
    p_j    = exp(s_j - max s) / sum_j' exp(s_j' - max s)
    out    = sum_j p_j v_j

Readings taken where the paper is silent:
  * K pool layout [num_blocks, Hkv, bs, D]; V pool layout [num_blocks, Hkv, D, bs]
    (the token index is fastest in V). The layout is part of the interface.
  * ctx_b counts the valid cached tokens (the new token's K/V already appended);
    table entries past ceil(ctx_b / bs) are never read; slots >= ctx_b of the
    last block are ignored.
  * An empty context (ctx_b = 0) gives out = 0.
"""
from __future__ import annotations

import math

import torch


def gather_sequence(k_cache, v_cache, block_table, b: int, ctx: int):
    """Logical K [Hkv, ctx, D] and V [Hkv, ctx, D] of sequence b, read through the table."""
    bs = k_cache.shape[2]
    j = torch.arange(ctx)
    phys = block_table[b].to(torch.int64)[j // bs]
    off = j % bs
    k = k_cache[phys, :, off, :]                 # [ctx, Hkv, D]
    v = v_cache[phys, :, :, off]                 # [ctx, Hkv, D]
    return k.permute(1, 0, 2).to(torch.float64), v.permute(1, 0, 2).to(torch.float64)


def attention_weights(q, k_cache, v_cache, block_table, context_lens, b: int, scale=None):
    """Softmax weights p [Hq, ctx_b] of sequence b (float64)."""
    Hq, D = q.shape[1], q.shape[2]
    Hkv = k_cache.shape[1]
    ctx = int(context_lens[b])
    if scale is None or scale == 0:
        scale = 1.0 / math.sqrt(D)
    k, _ = gather_sequence(k_cache, v_cache, block_table, b, ctx)
    group = torch.arange(Hq) // (Hq // Hkv)
    qb = q[b].to(torch.float64)                              # [Hq, D]
    s = torch.einsum("hd,hjd->hj", qb, k[group]) * scale     # [Hq, ctx]
    m = s.max(dim=1, keepdim=True).values
    e = torch.exp(s - m)
    return e / e.sum(dim=1, keepdim=True)


def attention_decode(q, k_cache, v_cache, block_table, context_lens, scale=None,
                     batch_indices=None):
    """out [B, Hq, D] float64 (rows not in ``batch_indices`` are left zero)."""
    B, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    assert Hq % Hkv == 0
    out = torch.zeros(B, Hq, D, dtype=torch.float64)
    group = torch.arange(Hq) // (Hq // Hkv)
    rows = range(B) if batch_indices is None else batch_indices
    for b in rows:
        ctx = int(context_lens[b])
        if ctx == 0:
            continue
        p = attention_weights(q, k_cache, v_cache, block_table, context_lens, b, scale)
        _, v = gather_sequence(k_cache, v_cache, block_table, b, ctx)
        out[b] = torch.einsum("hj,hjd->hd", p, v[group])
    return out
