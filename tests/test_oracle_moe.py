"""Pins of the top-k MoE oracle: library top-k, dense-mixture special case,
single-expert special case, routing-table invariants."""
import numpy as np
import torch
import torch.nn.functional as F

import oracle
from paper_2608_01891_amd import synth


def _dense_mixture(x, logits, w):
    """sum_e softmax(l)_e * SwiGLU_e(x) using torch library routines."""
    p = torch.softmax(logits.double(), dim=1)
    x = x.double()
    y = torch.zeros(x.shape[0], w.H, dtype=torch.float64)
    for e in range(w.E):
        ye = F.linear(F.silu(F.linear(x, w.w_gate[e].double())) * F.linear(x, w.w_up[e].double()),
                      w.w_down[e].double())
        y += p[:, e:e + 1] * ye
    return y


def test_k_equals_E_is_dense_softmax_mixture():
    x, w, logits = synth.custom_ffn(3, 6, 64, 96, E=4)
    y, ids, wt = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k=4)
    assert torch.allclose(y, _dense_mixture(x, logits, w), rtol=1e-12, atol=1e-15)


def test_single_expert_is_plain_swiglu():
    x, w, logits = synth.custom_ffn(4, 5, 64, 128, E=1)
    y, ids, wt = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k=1)
    assert torch.equal(ids, torch.zeros(5, 1, dtype=torch.int64))
    assert torch.equal(wt, torch.ones(5, 1, dtype=torch.float64))
    assert torch.equal(y, oracle.swiglu_ffn(x, w.w_gate[0], w.w_up[0], w.w_down[0]))


def test_topk_ids_match_stable_argsort_and_weights_match_softmax():
    rng = np.random.default_rng(3)
    logits = torch.from_numpy(rng.standard_normal((256, 8), dtype=np.float32))
    ids, w = oracle.route_topk(logits, 2)
    ref = np.argsort(-logits.numpy(), axis=1, kind="stable")[:, :2]
    assert np.array_equal(ids.numpy(), ref)
    sel = torch.gather(logits.double(), 1, ids)
    assert torch.allclose(w, torch.softmax(sel, dim=1), rtol=1e-15, atol=0)
    assert torch.allclose(w.sum(1), torch.ones(256, dtype=torch.float64), atol=1e-15)
    # equals the full softmax renormalised over the selected experts
    full = torch.softmax(logits.double(), dim=1)
    fsel = torch.gather(full, 1, ids)
    assert torch.allclose(w, fsel / fsel.sum(1, keepdim=True), rtol=1e-13)


def test_mixtral_workload_counts():
    rng = np.random.default_rng(3)
    logits = torch.from_numpy(rng.standard_normal((256, 8), dtype=np.float32))
    ids, _ = oracle.route_topk(logits, 2)
    counts, offsets, sorted_ids, pos = oracle.routing_tables(ids, 8)
    assert counts.tolist() == [62, 61, 76, 65, 63, 67, 56, 62]
    assert offsets.tolist() == [0] + np.cumsum([62, 61, 76, 65, 63, 67, 56, 62]).tolist()


def test_ties_go_to_lower_expert_id():
    logits = torch.tensor([[0.5, 2.0, 2.0, -1.0], [1.0, 1.0, 1.0, 1.0], [-0.0, 0.0, -3.0, 0.0]])
    ids, w = oracle.route_topk(logits, 2)
    assert ids.tolist() == [[1, 2], [0, 1], [0, 1]]
    assert torch.allclose(w[1], torch.tensor([0.5, 0.5], dtype=torch.float64))


def test_routing_tables_invariants():
    rng = np.random.default_rng(12)
    logits = torch.from_numpy(rng.standard_normal((37, 6), dtype=np.float32))
    ids, _ = oracle.route_topk(logits, 3)
    counts, offsets, sorted_ids, pos = oracle.routing_tables(ids, 6)
    assert int(counts.sum()) == 37 * 3
    assert sorted(sorted_ids.tolist()) == list(range(111))
    # independent order: numpy lexsort by (expert, pair id)
    flat = ids.reshape(-1).numpy()
    ref = np.lexsort((np.arange(111), flat))
    assert np.array_equal(sorted_ids.numpy(), ref)
    for e in range(6):
        seg = sorted_ids[offsets[e]:offsets[e + 1]]
        assert (ids.reshape(-1)[seg] == e).all()
    assert torch.equal(sorted_ids[pos], torch.arange(111))


def test_permute_unpermute_with_unit_weights_is_identity():
    rng = np.random.default_rng(13)
    logits = torch.from_numpy(rng.standard_normal((20, 5), dtype=np.float32))
    ids, _ = oracle.route_topk(logits, 2)
    _, _, sorted_ids, pos = oracle.routing_tables(ids, 5)
    x = torch.randn(20, 7, dtype=torch.float64)
    x_perm = x[sorted_ids // 2]
    back = sum(x_perm[pos.reshape(20, 2)[:, j]] for j in range(2)) / 2
    assert torch.equal(back, x)


def test_token_subset_matches_full():
    x, w, logits = synth.custom_ffn(5, 9, 64, 64, E=4)
    full, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k=2)
    sub, _, _ = oracle.moe_ffn(x, logits, w.w_gate, w.w_up, w.w_down, k=2, token_indices=[2, 7])
    assert torch.allclose(sub[[2, 7]], full[[2, 7]], rtol=1e-14, atol=1e-18)
    assert torch.equal(sub[0], torch.zeros(64, dtype=torch.float64))
