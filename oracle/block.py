"""Oracle: the steps on either side of decode attention in the attention stage
(float64 / exact copies).

Test infrastructure only (see the package docstring).

Each decode step appends the new token's key and value to the growing KV
cache before attending over it (the cache the paper's decode attention reads,
section 1 and section 2), and the attention output is projected back to the
hidden size before it crosses the A/F boundary (section 4.3: the attention
group sends its output to the FFN group).

    kv_append:  j = ctx_b - 1 (the new token is the last cached one)
                K[table[b, j // bs], g, j % bs, :] = k_new[b, g, :]
                V[table[b, j // bs], g, :, j % bs] = v_new[b, g, :]
    linear:     y = x W^T   (W in [out_features, in_features])

Readings: context_lens already counts the new token; sequences
with ctx_b = 0 append nothing; the projection has no bias.
"""
from __future__ import annotations

import torch


def kv_append(k_cache, v_cache, block_table, context_lens, k_new, v_new):
    """Copies of the two pools with each sequence's new token written in place."""
    k = k_cache.clone()
    v = v_cache.clone()
    bs = k.shape[2]
    for b in range(k_new.shape[0]):
        ctx = int(context_lens[b])
        if ctx == 0:
            continue
        j = ctx - 1
        p = int(block_table[b, j // bs])
        k[p, :, j % bs, :] = k_new[b]
        v[p, :, :, j % bs] = v_new[b]
    return k, v


def linear(x, w):
    """y [T, N] float64 for x [T, K], w [N, K]."""
    return x.to(torch.float64) @ w.to(torch.float64).T
