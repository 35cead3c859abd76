"""HIP KV append and linear projection vs the oracle (through the C ABI)."""
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.mark.parametrize("D,ctx", [(128, [1, 15, 16, 17, 32, 33, 700]), (64, [5, 16, 48, 200])])
def test_kv_append_bit_exact(gpu_lib, D, ctx):
    B = len(ctx)
    a = synth.custom_attention(95, B, 8, 2, D, ctx, ctx_hi=max(ctx) + 20)
    kn = synth.normal_tensor(95, 40, (B, 2, D))
    vn = synth.normal_tensor(95, 41, (B, 2, D))
    rk, rv = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, vn)
    ad = a.to(DEV)
    aflex.kv_append(ad, kn.to(DEV), vn.to(DEV))
    assert torch.equal(ad.k_cache.cpu(), rk) and torch.equal(ad.v_cache.cpu(), rv)


def test_kv_append_skips_empty_and_invalid(gpu_lib):
    a = synth.custom_attention(96, 3, 4, 2, 128, [0, 20, 40], ctx_hi=48)
    ad = a.to(DEV)
    bt = ad.block_table.clone()
    bt[2, 2] = -3  # the block of sequence 2's new token is invalid
    ad.block_table = bt
    k0, v0 = ad.k_cache.clone(), ad.v_cache.clone()
    kn = torch.full((3, 2, 128), 37.0, dtype=torch.bfloat16, device=DEV)
    aflex.kv_append(ad, kn, kn)
    ref_in = synth.AttnInputs(**{**a.__dict__})
    ref_in.context_lens = torch.tensor([0, 20, 0], dtype=torch.int32)
    rk, rv = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, ref_in.context_lens, kn.cpu(),
                              kn.cpu())
    assert torch.equal(ad.k_cache.cpu(), rk) and torch.equal(ad.v_cache.cpu(), rv)
    assert int((ad.k_cache != k0).sum()) == 2 * 128


def test_append_then_attention_matches_oracle(gpu_lib):
    a = synth.custom_attention(97, 4, 16, 2, 128, [1, 17, 300, 1000], ctx_hi=1024)
    kn = synth.normal_tensor(97, 40, (4, 2, 128))
    vn = synth.normal_tensor(97, 41, (4, 2, 128))
    ad = a.to(DEV)
    aflex.kv_append(ad, kn.to(DEV), vn.to(DEV))
    out = aflex.attn_decode(ad).cpu()
    rk, rv = oracle.kv_append(a.k_cache, a.v_cache, a.block_table, a.context_lens, kn, vn)
    check_rows(out, oracle.attention_decode(a.q, rk, rv, a.block_table, a.context_lens),
               what="append + attention")


@pytest.mark.parametrize("T,K,N", [(1, 64, 64), (7, 192, 320), (64, 256, 640), (300, 512, 448),
                                   (33, 1024, 128)])
def test_linear_shapes(gpu_lib, T, K, N):
    x = synth.normal_tensor(98, 4, (T, K))
    w = synth.normal_tensor(98, 8, (N, K), scale=0.02)
    y = aflex.linear(x.to(DEV), w.to(DEV)).cpu()
    check_rows(y, oracle.linear(x, w), what=f"linear T={T} K={K} N={N}")


@pytest.mark.parametrize("T,K,N", [(64, 8192, 5120), (256, 4096, 4096)])
def test_output_projection_shapes_all_rows(gpu_lib, T, K, N):
    """o_proj at the Qwen3-32B (64 x 8192 -> 5120) and Mixtral (256 x 4096 ->
    4096) decode shapes: every row."""
    x = synth.normal_tensor(99, 4, (T, K), device=DEV)
    w = synth.normal_tensor(99, 8, (N, K), scale=0.02, device=DEV)
    y = aflex.linear(x, w).cpu()
    check_rows(y, oracle.linear(x.cpu(), w.cpu()), what=f"o_proj T={T}")
