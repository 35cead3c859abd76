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
