"""Pins of the dense SwiGLU oracle."""
import math

import torch
import torch.nn.functional as F

import oracle
from paper_2608_01891_amd import synth


def test_scalar_closed_form():
    for x, wg, wu, wd in [(1.5, 0.7, -2.0, 3.0), (-4.0, 1.0, 1.0, 1.0), (0.25, -3.0, 5.0, -0.5)]:
        f = lambda v: torch.tensor([[v]], dtype=torch.float64)
        got = oracle.swiglu_ffn(f(x), f(wg), f(wu), f(wd))
        g = wg * x
        ref = wd * (g / (1 + math.exp(-g))) * (wu * x)
        assert abs(float(got) - ref) <= 1e-15 * max(1.0, abs(ref))


def test_zero_input_and_zero_up():
    x, w, _ = synth.custom_ffn(1, 3, 64, 96)
    assert torch.equal(oracle.swiglu_ffn(torch.zeros_like(x), w.w_gate, w.w_up, w.w_down),
                       torch.zeros(3, 64, dtype=torch.float64))
    assert torch.equal(oracle.swiglu_ffn(x, w.w_gate, torch.zeros_like(w.w_up), w.w_down),
                       torch.zeros(3, 64, dtype=torch.float64).abs())


def test_matches_torch_linear_and_silu():
    w = synth.tiny_layer()
    got = oracle.swiglu_ffn(w.x, w.ffn.w_gate, w.ffn.w_up, w.ffn.w_down)
    x = w.x.double()
    ref = F.linear(F.silu(F.linear(x, w.ffn.w_gate.double())) * F.linear(x, w.ffn.w_up.double()),
                   w.ffn.w_down.double())
    assert got.shape == (4, 512)
    assert torch.allclose(got, ref, rtol=1e-12, atol=1e-15)


def test_gate_and_up_are_not_interchangeable():
    # SiLU is applied to the gate projection only: swapping W_g and W_u changes y
    x, w, _ = synth.custom_ffn(2, 2, 64, 128)
    a = oracle.swiglu_ffn(x, w.w_gate, w.w_up, w.w_down)
    b = oracle.swiglu_ffn(x, w.w_up, w.w_gate, w.w_down)
    assert (a - b).abs().max() > 1e-3 * a.abs().max()


def test_silu_values():
    z = torch.tensor([0.0, 1.0, -1.0, 40.0, -40.0], dtype=torch.float64)
    s = oracle.silu(z)
    assert float(s[0]) == 0.0
    assert abs(float(s[1]) - 1 / (1 + math.exp(-1))) < 1e-16
    assert abs(float(s[2]) + 1 / (1 + math.exp(1))) < 1e-16
    assert abs(float(s[3]) - 40.0) < 1e-12 and abs(float(s[4])) < 1e-15
