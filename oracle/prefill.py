"""Oracle: causal prefill attention over packed variable-length prompts (float64).

Test infrastructure only (see the package docstring).

Prefill is the other phase of serving that the paper measures next to decode
(section 2 "LLM Serving"; section 3.2 contrasts how prefill and decode
attention follow the GPU clock): every prompt token attends to itself and to
the tokens before it in its own prompt. With prompts packed back to back
(cu[b] .. cu[b+1] - 1 are the tokens of prompt b) and i, j positions inside
prompt b:

    g        = h // (Hq // Hkv)                      (contiguous GQA groups)
    s_ij     = scale * <q[cu_b + i, h], k[cu_b + j, g]>,  j <= i
    p_ij     = exp(s_ij - max_j s_ij) / sum_j exp(s_ij - max_j s_ij)
    out[cu_b + i, h] = sum_{j <= i} p_ij v[cu_b + j, g]

Readings taken where the paper is silent: scale = 1/sqrt(D) unless given; the
mask is the standard causal one inside each prompt and nothing crosses prompt
boundaries; an empty prompt (cu[b] == cu[b+1]) produces no rows.
"""
from __future__ import annotations

import math

import torch


def attention_prefill(q, k, v, cu_seqlens, scale=None, rows=None):
    """out [T, Hq, D] float64 for q [T, Hq, D], k and v [T, Hkv, D].

    ``rows`` (optional) lists the token indices to compute; the others stay 0.
    """
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    assert Hq % Hkv == 0
    if scale is None or scale == 0:
        scale = 1.0 / math.sqrt(D)
    group = torch.arange(Hq) // (Hq // Hkv)
    out = torch.zeros(T, Hq, D, dtype=torch.float64)
    cu = [int(c) for c in cu_seqlens]
    want = None if rows is None else set(int(r) for r in rows)
    for b in range(len(cu) - 1):
        s0, s1 = cu[b], cu[b + 1]
        if s1 <= s0:
            continue
        kb = k[s0:s1].to(torch.float64)[:, group]   # [n, Hq, D]
        vb = v[s0:s1].to(torch.float64)[:, group]
        for i in range(s1 - s0):
            if want is not None and s0 + i not in want:
                continue
            qi = q[s0 + i].to(torch.float64)          # [Hq, D]
            s = torch.einsum("hd,jhd->hj", qi, kb[: i + 1]) * scale
            e = torch.exp(s - s.max(dim=1, keepdim=True).values)
            p = e / e.sum(dim=1, keepdim=True)
            out[s0 + i] = torch.einsum("hj,jhd->hd", p, vb[: i + 1])
    return out
