"""HIP top-k MoE FFN vs the oracle: routing indices bit-exact, values within
tolerance (through the C ABI)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.helpers import sample_rows
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _check_routing(r, logits, k, E):
    ids, w = oracle.route_topk(logits.cpu(), k)
    counts, offsets, sorted_ids, _ = oracle.routing_tables(ids, E)
    assert torch.equal(r["topk_ids"].cpu().long(), ids)
    assert torch.allclose(r["topk_w"].cpu().double(), w, rtol=2e-6, atol=1e-7)
    assert torch.equal(r["expert_offsets"].cpu().long(), offsets)
    assert torch.equal(r["sorted_pairs"].cpu().long(), sorted_ids)
    return ids


@pytest.mark.parametrize("T,H,I,E,k", [(37, 128, 192, 6, 3), (1, 64, 64, 8, 2), (100, 256, 320, 8, 2),
                                       (9, 128, 128, 4, 4), (12, 128, 64, 1, 1), (300, 192, 256, 16, 8),
                                       (400, 128, 192, 2, 1), (700, 192, 128, 3, 2)])
def test_small_shapes(gpu_lib, T, H, I, E, k):
    x, w, logits = synth.custom_ffn(60 + T, T, H, I, E=E)
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    _check_routing(r, logits, k, E)
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k)
    check_rows(y.cpu(), ref, what=f"moe T={T} E={E} k={k}")


def test_skewed_routing_all_to_one_expert(gpu_lib):
    T, H, I, E, k = 300, 128, 192, 8, 2
    x, w, logits = synth.custom_ffn(70, T, H, I, E=E)
    logits[:, 5] += 100.0  # every token picks expert 5 first: one segment of 300 rows
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    ids = _check_routing(r, logits, k, E)
    assert (ids[:, 0] == 5).all()
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k)
    check_rows(y.cpu(), ref, what="skewed moe")


def test_ties_in_logits(gpu_lib):
    T, H, I, E, k = 16, 64, 64, 4, 2
    x, w, _ = synth.custom_ffn(71, T, H, I, E=E)
    logits = torch.zeros(T, E)
    logits[::2, 3] = 1.0
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    ids = _check_routing(r, logits, k, E)
    assert ids[1].tolist() == [0, 1] and ids[0].tolist() == [3, 0]


def test_ties_and_infinities_across_logit_chunks(gpu_lib):
    """40 experts (the top-k pass reads logits 16 at a time): equal values
    across chunk boundaries keep the lower ids, -inf logits are taken only
    after every finite one, in id order."""
    T, H, I, E, k = 6, 64, 64, 40, 8
    x, w, _ = synth.custom_ffn(72, T, H, I, E=E)
    logits = torch.zeros(T, E)
    logits[0, [33, 17]] = 1.0
    logits[1, :] = float("-inf")
    logits[1, 30] = 0.0
    logits[2, :37] = float("-inf")
    logits[3, 15:18] = 2.0
    logits[4, ::5] = -1.0
    logits[5] = torch.arange(E, dtype=torch.float32).remainder(3)
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    ids = _check_routing(r, logits, k, E)
    assert ids[0].tolist() == [17, 33, 0, 1, 2, 3, 4, 5]
    assert ids[1].tolist() == [30, 0, 1, 2, 3, 4, 5, 6]
    assert ids[2].tolist() == [37, 38, 39, 0, 1, 2, 3, 4]
    assert ids[3].tolist() == [15, 16, 17, 0, 1, 2, 3, 4]
    assert ids[4].tolist() == [1, 2, 3, 4, 6, 7, 8, 9]
    assert ids[5].tolist() == [2, 5, 8, 11, 14, 17, 20, 23]


@pytest.fixture(scope="module")
def mixtral():
    wl = synth.mixtral_moe(device=DEV)
    yield wl
    del wl


def _tokens_of_every_pair_block(logits, k, E, block=256):
    """Tokens of the first and last (token, slot) pair of every block of
    ``block`` consecutive pairs in each expert's segment of the pair order:
    rows that cover every row tile of the grouped GEMMs."""
    ids, _ = oracle.route_topk(logits.cpu(), k)
    _, offsets, sorted_ids, _ = oracle.routing_tables(ids, E)
    toks = set()
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        for p0 in range(lo, hi, block):
            for p in (p0, min(p0 + block, hi) - 1):
                toks.add(int(sorted_ids[p]) // k)
    return sorted(toks)


def test_mixtral_shape_all_rows(gpu_lib, mixtral):
    wl = mixtral
    y, r = aflex.moe_ffn(wl.x, wl.ffn, wl.router_logits, 2, routing=True)
    ids = _check_routing(r, wl.router_logits, 2, 8)
    counts = torch.bincount(ids.reshape(-1), minlength=8)
    assert counts.tolist() == [62, 61, 76, 65, 63, 67, 56, 62]
    y = y.cpu()
    f = wl.ffn
    ref, _, _ = oracle.moe_ffn(wl.x.cpu(), wl.router_logits.cpu(), f.w_gate.cpu(), f.w_up.cpu(),
                               f.w_down.cpu(), 2)
    check_rows(y, ref, what="mixtral moe T=256 (all rows)")
    y2 = aflex.moe_ffn(wl.x, wl.ffn, wl.router_logits, 2).cpu()
    assert torch.equal(y, y2)


def test_mixtral_2048_tokens_all_rows(gpu_lib, mixtral):
    """The MoE at 2048 tokens (seed 103), the MFMA-bound decode size timed by the
    benchmark (256-row tiles, routing in three kernels): every row."""
    T = 2048
    wl = synth.mixtral_moe(device=DEV, T=T, seed=103, weights=mixtral.ffn)
    y, r = aflex.moe_ffn(wl.x, wl.ffn, wl.router_logits, 2, routing=True)
    _check_routing(r, wl.router_logits, 2, 8)
    f = wl.ffn
    ref, _, _ = oracle.moe_ffn(wl.x.cpu(), wl.router_logits.cpu(), f.w_gate.cpu(), f.w_up.cpu(),
                               f.w_down.cpu(), 2)
    check_rows(y.cpu(), ref, what="mixtral moe T=2048 (all rows)")


def test_mixtral_prefill_tokens_every_row_tile(gpu_lib, mixtral):
    """The MoE FFN over a prefill batch (T = 4096 tokens, 8192 token/slot
    pairs): the tokens of the first and last pair of every 256-pair block of
    each expert, plus random tokens."""
    T = 4096
    wl = synth.mixtral_moe(device=DEV, T=T, seed=7, weights=mixtral.ffn)
    y, r = aflex.moe_ffn(wl.x, wl.ffn, wl.router_logits, 2, routing=True)
    _check_routing(r, wl.router_logits, 2, 8)
    edges = _tokens_of_every_pair_block(wl.router_logits, 2, 8)
    toks = sample_rows(T, len(edges) + 8, seed=7, must=edges + [0, T - 1])
    f = wl.ffn
    ref, _, _ = oracle.moe_ffn(wl.x.cpu(), wl.router_logits.cpu(), f.w_gate.cpu(), f.w_up.cpu(),
                               f.w_down.cpu(), 2, token_indices=toks)
    check_rows(y.cpu()[toks], ref[toks], what="mixtral moe prefill T=4096 (every pair block)")


@pytest.mark.parametrize("T,E,k", [(200, 64, 8), (33, 64, 1), (64, 2, 2), (512, 8, 2), (513, 8, 2),
                                   (1025, 3, 3), (1500, 64, 8), (2000, 64, 1)])
def test_routing_extremes(gpu_lib, T, E, k):
    """The largest supported expert count and top-k (E = 64, k = 8), top-1 over
    64 experts (many empty experts), and k = E; on both sides of the batch size
    where routing moves from one work-group to one per 256 tokens (512), with
    ragged last chunks."""
    H, I = 128, 128
    x, w, logits = synth.custom_ffn(80 + E + k, T, H, I, E=E)
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    _check_routing(r, logits, k, E)
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k)
    check_rows(y.cpu(), ref, what=f"moe extremes T={T} E={E} k={k}")


@pytest.mark.parametrize("T", [20, 160, 200, 384, 448, 576, 584, 600, 1024, 1200, 2048, 2500])
def test_tile_shape_boundaries(gpu_lib, T):
    """Average rows per expert on both sides of the tile-size thresholds with 8
    experts and top-2: 32-row tiles (5), 64-row (40), 128-row with
    non-temporal weights (50, 96), 128-row re-reading weights (112, 144),
    256-row tiles (146, 150, 300, 625) and 320-row tiles (256, 512; experts
    of either side of 320 and 640 rows)."""
    x, w, logits = synth.custom_ffn(90 + T, T, 256, 192, E=8)
    y = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), 2).cpu()
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, 2)
    check_rows(y, ref, what=f"moe tile boundary T={T}")


@pytest.mark.parametrize("T,H,I,E,k", [(16, 128, 8192, 4, 3),     # 32-row tiles, 8 splits, k > 2
                                       (24, 128, 5120, 4, 2),     # 5 splits: a second, partly used batch
                                       (200, 128, 8192, 2, 2)])   # 256-row tiles, split count planned on the device
def test_many_down_splits(gpu_lib, T, H, I, E, k):
    """Narrow H and wide I give the down GEMM many K splits, so the combine sums
    its partials over more than one batch of four splits (and over k > 2
    pairs) before weighting them."""
    x, w, logits = synth.custom_ffn(90 + T, T, H, I, E=E)
    y, r = aflex.moe_ffn(x.to(DEV), w.to(DEV), logits.to(DEV), k, routing=True)
    _check_routing(r, logits, k, E)
    ref, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k)
    check_rows(y.cpu(), ref, what=f"moe many splits T={T} I={I} k={k}")
