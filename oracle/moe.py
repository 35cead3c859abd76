"""Oracle: top-k mixture-of-experts SwiGLU FFN (float64 values, exact indices).

Test infrastructure only (see the package docstring).

The paper's MoE model is Mixtral-8x7B (section 6.1); sparse expert execution
changes the FFN's computation and communication (section 6.2, "Generality").
For each token t with router logits l_t[0..E):

    ids_t  = the k experts ordered by (logit descending, expert id ascending)
    w_t,j  = exp(l_t[ids_j]) / sum_{j'<k} exp(l_t[ids_j'])     (softmax over the k)
    y_t    = sum_{j<k} w_t,j * SwiGLU_{ids_j}(x_t)              (in slot order)

Routing tables (the index work of the permute/un-permute steps):
    counts[e]   = number of (token, slot) pairs routed to e
    offsets     = exclusive prefix sum of counts, length E+1
    sorted      = pair ids t*k+j ordered by (expert, token, slot)
    position    = inverse of sorted: position[t*k+j] = rank of that pair

Readings taken where the paper is silent: logits are fp32 and widened exactly, so the
ordering is the fp32 ordering; ties go to the lower expert id; the weights are
the softmax over the selected logits, which equals the full softmax
renormalised over the top-k.
"""
from __future__ import annotations

import torch

from .ffn import swiglu_ffn


def route_topk(logits: torch.Tensor, k: int):
    """ids [T, k] int64 and weights [T, k] float64."""
    T, E = logits.shape
    l64 = logits.to(torch.float64)
    ids = torch.empty(T, k, dtype=torch.int64)
    w = torch.empty(T, k, dtype=torch.float64)
    for t in range(T):
        row = [float(v) for v in l64[t]]
        order = sorted(range(E), key=lambda e: (-row[e], e))[:k]
        ids[t] = torch.tensor(order)
        sel = l64[t, ids[t]]
        e = torch.exp(sel - sel.max())
        w[t] = e / e.sum()
    return ids, w


def routing_tables(ids: torch.Tensor, E: int):
    """counts [E], offsets [E+1], sorted pair ids [T*k], position [T*k] (all int64)."""
    T, k = ids.shape
    pairs = [(int(ids[t, j]), t, j) for t in range(T) for j in range(k)]
    order = sorted(pairs)
    counts = torch.zeros(E, dtype=torch.int64)
    for e, _, _ in pairs:
        counts[e] += 1
    offsets = torch.zeros(E + 1, dtype=torch.int64)
    offsets[1:] = torch.cumsum(counts, 0)
    sorted_ids = torch.tensor([t * k + j for _, t, j in order], dtype=torch.int64)
    position = torch.empty(T * k, dtype=torch.int64)
    position[sorted_ids] = torch.arange(T * k)
    return counts, offsets, sorted_ids, position


def moe_ffn(x, logits, w_gate, w_up, w_down, k: int, token_indices=None):
    """y [T, H] float64, ids [T, k], w [T, k].

    Each expert's SwiGLU is evaluated once on the tokens routed to it (rows are
    independent, so this is the per-token definition); the k expert outputs of
    a token are then summed in slot order. ``token_indices`` restricts the
    expert evaluation to those tokens (other rows of y stay zero); the routing
    is always computed for every token.
    """
    T, H = x.shape
    E = logits.shape[1]
    ids, w = route_topk(logits, k)
    rows = list(range(T)) if token_indices is None else [int(t) for t in token_indices]
    expert_out = {}
    for e in range(E):
        sel = [(t, j) for t in rows for j in range(k) if int(ids[t, j]) == e]
        if not sel:
            continue
        toks = torch.tensor([t for t, _ in sel], dtype=torch.int64)
        ye = swiglu_ffn(x[toks], w_gate[e], w_up[e], w_down[e])
        for r, key in enumerate(sel):
            expert_out[key] = ye[r]
    y = torch.zeros(T, H, dtype=torch.float64)
    for t in rows:
        acc = torch.zeros(H, dtype=torch.float64)
        for j in range(k):
            acc = acc + w[t, j] * expert_out[(t, j)]
        y[t] = acc
    return y, ids, w
