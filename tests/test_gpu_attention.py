"""HIP decode attention vs the oracle (through the C ABI)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _oracle(a, rows=None):
    return oracle.attention_decode(a.q, a.k_cache, a.v_cache, a.block_table, a.context_lens,
                                   batch_indices=rows)


def test_tiny_layer(gpu_lib):
    w = synth.tiny_layer()
    out = aflex.attn_decode(w.attn.to(DEV)).cpu()
    check_rows(out, _oracle(w.attn), what="tiny-layer attention")


@pytest.mark.parametrize("D,Hq,Hkv,split", [(128, 16, 2, 128), (128, 8, 1, 256), (64, 32, 2, 128),
                                            (64, 4, 4, 0), (128, 64, 8, 384)])
def test_ragged_multi_split(gpu_lib, D, Hq, Hkv, split):
    ctx = [1, 15, 16, 17, 31, 33, 600, 1300, 127, 129]
    a = synth.custom_attention(31, len(ctx), Hq, Hkv, D, ctx, ctx_hi=1400)
    out = aflex.attn_decode(a.to(DEV), split_tokens=split).cpu()
    check_rows(out, _oracle(a), what=f"ragged D={D} G={Hq // Hkv} split={split}")


@pytest.mark.parametrize("split", [1024, 0])
def test_full_1024_token_splits(gpu_lib, split):
    """Splits of 64 blocks (every lane of a wave holds a block id), exact and
    ragged multiples of the split, with 8 query heads per KV head."""
    ctx = [1024, 1025, 2047, 2048, 3000, 5, 64, 4100]
    a = synth.custom_attention(32, len(ctx), 64, 8, 128, ctx, ctx_hi=4200)
    out = aflex.attn_decode(a.to(DEV), split_tokens=split).cpu()
    check_rows(out, _oracle(a), what=f"1024-token splits (split={split})")


@pytest.mark.parametrize("seed", [0, 1])
def test_many_short_units_partition(gpu_lib, seed):
    """Hundreds of short (sequence, kv head) units between empty sequences and a
    few long ones: the even split charges every unit a fixed cost besides its
    blocks, so work-group ranges start and end inside units, inside a unit's
    charge (no block of it) and across runs of empty sequences."""
    rng = np.random.default_rng(900 + seed)
    ctx = rng.integers(1, 49, 300)
    ctx[rng.random(300) < 0.2] = 0
    ctx[rng.choice(300, 4, replace=False)] = rng.integers(2000, 6000, 4)
    a = synth.custom_attention(40 + seed, len(ctx), 32, 8, 128, ctx, ctx_hi=6000)
    out = aflex.attn_decode(a.to(DEV)).cpu()
    ref = _oracle(a)
    nz = torch.from_numpy(ctx > 0)
    check_rows(out[nz], ref[nz], what=f"many short units (seed {seed})")
    assert torch.count_nonzero(out[~nz]) == 0


@pytest.mark.parametrize("B,Hkv,hi", [(96, 8, 512), (5, 2, 40), (97, 8, 512)])
def test_short_contexts_one_unit_per_work_group(gpu_lib, B, Hkv, hi):
    """Contexts up to 512 tokens with every (sequence, kv head) unit in one
    round of resident work-groups (96 x 8 units on 768) take one work-group per
    unit and no merge launch; 97 x 8 units fall back to the even split."""
    rng = np.random.default_rng(950 + B)
    ctx = rng.integers(1, hi + 1, B)
    ctx[rng.random(B) < 0.15] = 0
    ctx[0] = hi
    a = synth.custom_attention(60 + B, B, 4 * Hkv, Hkv, 128, ctx, ctx_hi=hi)
    out = aflex.attn_decode(a.to(DEV)).cpu()
    nz = torch.from_numpy(ctx > 0)
    check_rows(out[nz], _oracle(a)[nz], what=f"short contexts B={B} Hkv={Hkv}")
    assert torch.count_nonzero(out[~nz]) == 0


def test_qwen3_shape_all_rows(gpu_lib):
    """The Qwen3-32B workload at full size (B = 64, 64/8 heads, lognormal
    contexts): every sequence and head against the oracle."""
    w = synth.qwen3_attention(device=DEV)
    a = w.attn
    out = aflex.attn_decode(a).cpu()
    check_rows(out, _oracle(a.to("cpu")), what="qwen3 attention (all 64 sequences)")


def test_long_context_shape_all_rows(gpu_lib):
    """The pipeline workload's attention at full size (B = 256, 32/8 heads,
    contexts up to 22384 tokens, 1024-token splits): every row."""
    w = synth.af_pipeline(device=DEV)
    a = w.attn
    out = aflex.attn_decode(a).cpu()
    check_rows(out, _oracle(a.to("cpu")), what="long-context attention (all 256 sequences)")


def test_context_one_is_v_bitwise(gpu_lib):
    a = synth.custom_attention(40, 5, 16, 2, 128, [1, 1, 1, 1, 1], ctx_hi=64)
    out = aflex.attn_decode(a.to(DEV)).cpu()
    for b in range(5):
        p = int(a.block_table[b, 0])
        for h in range(16):
            assert torch.equal(out[b, h], a.v_cache[p, h // 8, :, 0]), (b, h)


def test_equal_v_rows_bitwise(gpu_lib):
    a = synth.custom_attention(41, 3, 8, 2, 128, [700, 33, 260], ctx_hi=800)
    v = a.v_cache.clone()
    row = synth.normal_tensor(41, 99, (2, 128))
    v[:] = row[None, :, :, None]
    a.v_cache = v
    out = aflex.attn_decode(a.to(DEV), split_tokens=256).cpu()
    for b in range(3):
        for h in range(8):
            assert torch.equal(out[b, h], row[h // 4]), (b, h)


def test_empty_context_and_clamped_length(gpu_lib):
    a = synth.custom_attention(42, 3, 8, 2, 64, [0, 45, 320], ctx_hi=320)
    ad = a.to(DEV)
    ad.context_lens = torch.tensor([0, 45, 5000], dtype=torch.int32, device=DEV)  # > max_context_len
    out = aflex.attn_decode(ad).cpu()
    assert torch.equal(out[0], torch.zeros(8, 64, dtype=torch.bfloat16))
    ref = a
    ref.context_lens = torch.tensor([0, 45, 320], dtype=torch.int32)
    check_rows(out[1:], _oracle(ref)[1:], what="clamped context")


def test_nan_poisoned_tails_and_unused_blocks_do_not_leak(gpu_lib):
    a = synth.custom_attention(43, 4, 8, 2, 128, [17, 250, 33, 1], ctx_hi=256)
    ref = _oracle(a)
    k = a.k_cache.clone(); v = a.v_cache.clone()
    for b, c in enumerate(a.context_lens.tolist()):
        last = int(a.block_table[b, (c - 1) // 16])
        if c % 16:
            k[last, :, c % 16:, :] = float("nan")
            v[last, :, :, c % 16:] = float("nan")
    # extra pool blocks no table entry points at
    k = torch.cat([k, torch.full((3,) + tuple(k.shape[1:]), float("nan"), dtype=k.dtype)])
    v = torch.cat([v, torch.full((3,) + tuple(v.shape[1:]), float("nan"), dtype=v.dtype)])
    a.k_cache, a.v_cache, a.num_blocks = k, v, a.num_blocks + 3
    out = aflex.attn_decode(a.to(DEV)).cpu()
    check_rows(out, ref, what="NaN-poisoned tails")


def test_out_of_range_block_ids_are_skipped(gpu_lib):
    # an invalid id in the last table slot of a sequence masks that block's tokens
    a = synth.custom_attention(44, 2, 8, 2, 128, [40, 64], ctx_hi=64)
    ad = a.to(DEV)
    bt = ad.block_table.clone()
    bt[0, 2] = a.num_blocks + 7
    bt[1, 3] = -5
    ad.block_table = bt
    out = aflex.attn_decode(ad).cpu()
    ref_in = a
    ref_in.context_lens = torch.tensor([32, 48], dtype=torch.int32)
    check_rows(out, _oracle(ref_in), what="out-of-range block ids")


def test_inputs_unmodified_and_deterministic(gpu_lib):
    w = synth.qwen3_attention(device=DEV)
    a = w.attn
    bt0, cl0, q0 = a.block_table.clone(), a.context_lens.clone(), a.q.clone()
    o1 = aflex.attn_decode(a)
    o2 = aflex.attn_decode(a)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    assert torch.equal(a.block_table, bt0) and torch.equal(a.context_lens, cl0)
    assert torch.equal(a.q, q0)


def test_generator_bits_match_cpu(gpu_lib):
    idx = torch.randint(0, 1 << 31, (4096,), dtype=torch.int64)
    for s in (1, 2, 3, 5, 7):
        cpu = synth.normal_at(4, s, idx, scale=0.02 if s >= 5 else 1.0)
        gpu = synth.normal_at(4, s, idx.to(DEV), scale=0.02 if s >= 5 else 1.0).cpu()
        assert torch.equal(cpu, gpu)
