"""Comparison helpers for HIP-vs-oracle parity (test code only).

Tolerance (bf16 inputs, fp32 accumulation, bf16 outputs): max relative error
2e-2, applied two ways, both of which must hold for every row (a row is one
(sequence, head) for attention and one token for the FFNs):
  * row-normwise:  max_i |y_i - r_i| <= 2e-2 * max_i |r_i|
  * elementwise:   |y_i - r_i| <= 2e-2 * |r_i| + 2e-2 * rms(r_row)
"""
import torch

RTOL = 2e-2


def check_rows(y, ref, rtol=RTOL, what=""):
    y = y.to(torch.float64).reshape(-1, y.shape[-1])
    ref = ref.to(torch.float64).reshape(-1, ref.shape[-1])
    assert y.shape == ref.shape, (y.shape, ref.shape)
    assert torch.isfinite(y).all(), f"{what}: non-finite output"
    err = (y - ref).abs()
    rmax = ref.abs().amax(dim=1)
    rms = ref.pow(2).mean(dim=1).sqrt()
    norm_ok = err.amax(dim=1) <= rtol * rmax + 1e-30
    elem_ok = (err <= rtol * ref.abs() + rtol * rms[:, None] + 1e-30).all(dim=1)
    bad = (~norm_ok) | (~elem_ok)
    if bad.any():
        i = int(bad.nonzero()[0])
        raise AssertionError(
            f"{what}: {int(bad.sum())} rows out of tolerance; first row {i}: "
            f"max err {float(err[i].max()):.3e} vs max|ref| {float(rmax[i]):.3e}")
    return float((err.amax(dim=1) / rmax.clamp_min(1e-30)).max())
