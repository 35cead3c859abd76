"""Oracle: dense SwiGLU FFN (float64).

Test infrastructure only (see the package docstring).

The FFN is the operator the paper finds memory-bound at small decode batches
and compute-bound, hence clock-sensitive, at large ones (section 1; section 3.2
reports a 71.5% decode latency change over the clock range). For the dense
model it evaluates (Qwen3-32B, section 6.1) the FFN is SwiGLU:

    g = x W_g^T,  u = x W_u^T,  h = SiLU(g) * u,  y = h W_d^T
    SiLU(z) = z / (1 + exp(-z))

Weights follow the [out_features, in_features] convention: W_g, W_u are
[I, H] and W_d is [H, I]. The intermediate h is kept in float64 (no rounding).
"""
from __future__ import annotations

import torch


def silu(z: torch.Tensor) -> torch.Tensor:
    return z / (1.0 + torch.exp(-z))


def swiglu_ffn(x, w_gate, w_up, w_down) -> torch.Tensor:
    """y [T, H] float64 for x [T, H]."""
    x = x.to(torch.float64)
    g = x @ w_gate.to(torch.float64).T
    u = x @ w_up.to(torch.float64).T
    h = silu(g) * u
    return h @ w_down.to(torch.float64).T
