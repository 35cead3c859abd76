"""HIP MoE block (RMSNorm + router GEMM + top-k MoE) vs the oracle.

The router logits are computed on both sides, so a routing decision is unique
only where the top-k margin exceeds the logits' rounding error: those tokens
must route identically and match the oracle's output; for the rest (near
ties) the GPU's choice must be a valid top-k of its own logits.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
MARGIN = 1e-3


def _inputs(seed, T, H, I, E):
    x, w, _ = synth.custom_ffn(seed, T, H, I, E=E)
    gamma = (1.0 + 0.1 * synth.normal_tensor(seed, 50, (H,), dtype=torch.float32)).to(torch.bfloat16)
    wr = synth.normal_tensor(seed, 51, (E, H), scale=0.02)
    return x, w, gamma, wr


def _margins(logits, k):
    s = torch.sort(logits.double(), dim=1, descending=True).values
    gaps = s[:, :k] - s[:, 1:k + 1]  # gaps between consecutive ranks down to the (k+1)-th
    return gaps.min(dim=1).values


def _check(y, lg, r, ref_y, ref_lg, ref_ids, k, rows=None):
    lg, ids = lg.cpu().double(), r["topk_ids"].cpu().long()
    scale = ref_lg.abs().amax(dim=1, keepdim=True)
    assert ((lg - ref_lg).abs() <= 1e-5 * scale + 1e-6).all()
    clear = _margins(ref_lg, k) > MARGIN
    assert torch.equal(ids[clear], ref_ids[clear])
    for t in (~clear).nonzero().flatten().tolist():  # near ties: a valid top-k of the GPU logits
        own = np.argsort(-lg[t].numpy(), kind="stable")[:k]
        assert sorted(own.tolist()) == sorted(ids[t].tolist())
    assert int((~clear).sum()) <= max(2, clear.numel() // 20)
    keep = [t for t in (rows if rows is not None else range(clear.numel())) if bool(clear[t])]
    check_rows(y.cpu()[keep], ref_y[keep], what="moe block")


@pytest.mark.parametrize("T,H,I,E,k,res", [(37, 128, 192, 6, 3, False), (64, 256, 128, 8, 2, True),
                                           (5, 512, 256, 4, 1, True), (9, 2048, 128, 16, 2, False),
                                           (3, 8192, 128, 8, 2, True), (2, 16384, 64, 20, 4, False)])
def test_small_shapes(gpu_lib, T, H, I, E, k, res):
    x, w, gamma, wr = _inputs(120 + T, T, H, I, E)
    y, lg, r = aflex.moe_block(x.to(DEV), w.to(DEV), gamma.to(DEV), wr.to(DEV), k, eps=1e-5,
                               residual=res, routing=True)
    ref_y, ref_lg, ref_ids = oracle.moe_block(x, gamma, 1e-5, wr, w.w_gate, w.w_up, w.w_down, k, res)
    _check(y, lg, r, ref_y, ref_lg, ref_ids, k)


def test_mixtral_shape_all_rows(gpu_lib):
    T, H, I, E, k = 256, 4096, 14336, 8, 2
    x, _, _ = synth.custom_ffn(130, T, H, 64, E=E)
    w = synth.make_ffn_weights(130, H, I, E, device=DEV)
    gamma = (1.0 + 0.1 * synth.normal_tensor(130, 50, (H,), dtype=torch.float32)).to(torch.bfloat16)
    wr = synth.normal_tensor(130, 51, (E, H), scale=0.02)
    y, lg, r = aflex.moe_block(x.to(DEV), w, gamma.to(DEV), wr.to(DEV), k, eps=1e-5, residual=True,
                               routing=True)
    ref_y, ref_lg, ref_ids = oracle.moe_block(x, gamma, 1e-5, wr, w.w_gate.cpu(), w.w_up.cpu(),
                                              w.w_down.cpu(), k, True)
    _check(y, lg, r, ref_y, ref_lg, ref_ids, k)
