"""Oracle: the steps on either side of decode attention in the attention stage
(float64 / exact copies).

Test infrastructure only (see the package docstring).

Each decode step appends the new token's key and value to the growing KV
cache before attending over it (the cache the paper's decode attention reads,
section 1 and section 2), and the attention output is projected back to the
hidden size before it crosses the A/F boundary (section 4.3: the attention
group sends its output to the FFN group).

The FFN stage of the MoE model starts the same way on the F side: the
Mixtral layer normalises the hidden state (RMSNorm) and computes the router
logits before the experts run (section 6.1 names the model):

    kv_append:  j = ctx_b - 1 (the new token is the last cached one)
                K[table[b, j // bs], g, j % bs, :] = k_new[b, g, :]
                V[table[b, j // bs], g, :, j % bs] = v_new[b, g, :]
    kv_write:   the same for n_b new tokens per sequence (a prefilled prompt,
                section 2: prefill populates the KV cache), j = ctx_b - n_b + i
    linear:     y = x W^T   (W in [out_features, in_features])
    rmsnorm:    x / sqrt(mean(x^2) + eps) * gamma
    moe_block:  y = MoE(RMSNorm(x), RMSNorm(x) W_r^T) (+ x with the residual)

Readings taken where the paper is silent: context_lens already counts the new token; sequences
with ctx_b = 0 append nothing; the projection has no bias.
"""
from __future__ import annotations

import torch

from .moe import moe_ffn


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


def kv_write(k_cache, v_cache, block_table, context_lens, cu_seqlens, k_new, v_new):
    """Copies of the two pools with each sequence's new tokens written at the end
    of its context: rows cu[b] .. cu[b+1]-1 of k_new / v_new are the n_b newest
    tokens of sequence b, so token i lands at position ctx_b - n_b + i. A prompt
    written by prefill has ctx_b = n_b (positions 0 .. n_b-1); one decode token
    per sequence (n_b = 1) is kv_append. Positions below 0 (ctx_b < n_b) are not
    written."""
    k = k_cache.clone()
    v = v_cache.clone()
    bs = k.shape[2]
    cu = [int(c) for c in cu_seqlens]
    for b in range(len(cu) - 1):
        n = cu[b + 1] - cu[b]
        ctx = int(context_lens[b])
        for i in range(n):
            j = ctx - n + i
            if j < 0:
                continue
            p = int(block_table[b, j // bs])
            k[p, :, j % bs, :] = k_new[cu[b] + i]
            v[p, :, :, j % bs] = v_new[cu[b] + i]
    return k, v


def linear(x, w):
    """y [T, N] float64 for x [T, K], w [N, K]."""
    return x.to(torch.float64) @ w.to(torch.float64).T


def rmsnorm(x, gamma, eps: float):
    """x / sqrt(mean(x^2) + eps) * gamma over the last dimension (float64)."""
    x = x.to(torch.float64)
    inv = 1.0 / torch.sqrt((x * x).mean(dim=-1, keepdim=True) + eps)
    return x * inv * gamma.to(torch.float64)


def moe_block(x, gamma, eps: float, w_router, w_gate, w_up, w_down, k: int, residual: bool,
              token_indices=None):
    """The MoE FFN block of a Mixtral layer: normalise, route, mix experts.

        xn     = RMSNorm(x)
        logits = xn W_r^T                       (W_r [E, H])
        y      = MoE(xn, logits) (+ x if residual)

    Returns y [T, H], logits [T, E], ids [T, k] (float64 / int64).
    """
    xn = rmsnorm(x, gamma, eps)
    logits = xn @ w_router.to(torch.float64).T
    y, ids, _ = moe_ffn(xn, logits, w_gate, w_up, w_down, k, token_indices=token_indices)
    if residual:
        y = y + x.to(torch.float64)
    return y, logits, ids
