"""Oracle: the interleaved A/F decode layer step, as plain serial composition (float64).

Test infrastructure only (see the package docstring).

The paper's data plane runs each transformer layer as a two-stage A->F
pipeline over M microbatches; A_{l+1,i} may start as soon as F_{l,i} is done
(section 4.3, "Interleaved A/F Pipeline"; Eq. 2 models its timing). Both
stages are row-independent, so whatever the schedule, the values are those of
running, for every microbatch i and layer l in order,

    a   = Attention(q_i)                    [n_i, Hq, D]
    y   = FFN(a viewed as [n_i, Hq*D])      (dense SwiGLU, or top-k MoE with
                                             microbatch i's router logits)
    q_i = y viewed as [n_i, Hq, D]          (input of the next layer step)

Readings taken where the paper is silent: the attention output feeds the FFN directly (no output
projection or normalisation, which lie outside the operator pair); later layer
steps reuse the same KV cache and weights; microbatches are contiguous slices
of the batch in order.
"""
from __future__ import annotations

import torch

from .attention import attention_decode
from .block import kv_append, linear, moe_block
from .ffn import swiglu_ffn
from .moe import moe_ffn


def af_layer_steps(attn, ffn, router_logits, top_k: int, mb_sizes, L: int = 1):
    """y [B, Hq*D] float64 after L layer steps, microbatch by microbatch."""
    B, Hq, D = attn.q.shape
    H = Hq * D
    assert sum(mb_sizes) == B
    out = torch.zeros(B, H, dtype=torch.float64)
    start = 0
    for n in mb_sizes:
        sl = slice(start, start + n)
        q = attn.q[sl].to(torch.float64)
        for _ in range(L):
            a = attention_decode(q, attn.k_cache, attn.v_cache, attn.block_table[sl],
                                 attn.context_lens[sl])
            a = a.reshape(n, H)
            if ffn.E:
                y, _, _ = moe_ffn(a, router_logits[sl], ffn.w_gate, ffn.w_up, ffn.w_down, top_k)
            else:
                y = swiglu_ffn(a, ffn.w_gate, ffn.w_up, ffn.w_down)
            q = y.reshape(n, Hq, D)
        out[sl] = q.reshape(n, H)
        start += n
    return out


def af_decode_layer_steps(attn, ffn, layer, top_k: int, mb_sizes, L: int = 1):
    """The whole decode layer on the A/F step (section 4.3: the attention group
    runs attention and sends its output to the FFN group), microbatch by
    microbatch, float64. With K', V' the pools after appending each sequence's
    new token (kv_append) and, for microbatch i,

        a   = Attention(q_i over K', V')             [n_i, Hq*D]
        h   = a W_o^T (+ x_i)                        (x_i: layer input rows, if given)
        y   = h + MoE(RMSNorm(h), RMSNorm(h) W_r^T)  (moe_block with the residual)
        q_i, x_i = y viewed [n_i, Hq, D], y          (input of the next layer step)

    Returns y [B, H] after L steps and the router logits of every step
    (a list of L tensors [B, E]). Later steps would append the same token to
    the same slot again, which leaves the pools as they are, so the pools
    are appended once.
    """
    B, Hq, D = attn.q.shape
    H = ffn.H
    assert sum(mb_sizes) == B
    kc, vc = kv_append(attn.k_cache, attn.v_cache, attn.block_table, attn.context_lens,
                       layer.k_new, layer.v_new)
    out = torch.zeros(B, H, dtype=torch.float64)
    logits = [torch.zeros(B, ffn.E, dtype=torch.float64) for _ in range(L)]
    start = 0
    for n in mb_sizes:
        sl = slice(start, start + n)
        q = attn.q[sl].to(torch.float64)
        x = None if layer.x_in is None else layer.x_in[sl].to(torch.float64)
        for step in range(L):
            a = attention_decode(q, kc, vc, attn.block_table[sl], attn.context_lens[sl])
            h = linear(a.reshape(n, Hq * D), layer.w_o)
            if x is not None:
                h = h + x
            y, lg, _ = moe_block(h, layer.norm_weight, layer.eps, layer.router_weight, ffn.w_gate,
                                 ffn.w_up, ffn.w_down, top_k, residual=True)
            logits[step][sl] = lg
            q, x = y.reshape(n, Hq, D), y
        out[sl] = y
        start += n
    return out, logits
