"""HIP causal prefill attention vs the oracle (through the C ABI)."""
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _run(p, **kw):
    return aflex.attn_prefill(p.to(DEV), **kw).cpu()


@pytest.mark.parametrize("lens,Hq,Hkv", [
    ([1, 5, 0, 130, 64, 200], 8, 2),        # empty prompt, one-token prompt, ragged tails
    ([63, 64, 65, 127, 128, 129], 8, 8),    # tile edges, MHA
    ([300], 16, 1),                         # 16 query heads on one KV head
    ([257, 3], 12, 4),                      # Hq not a multiple of 8 (no head permutation)
    ([0, 0, 17], 32, 8),
])
def test_small_shapes(gpu_lib, lens, Hq, Hkv):
    p = synth.make_prefill(40 + len(lens), lens, Hq, Hkv, 128)
    out = _run(p)
    ref = oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens)
    check_rows(out, ref, what=f"prefill lens={lens} Hq={Hq} Hkv={Hkv}")


def test_one_long_prompt_full(gpu_lib):
    p = synth.make_prefill(47, [1000], 8, 2, 128)
    out = _run(p)
    check_rows(out, oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens), what="prefill n=1000")


def test_scale_argument(gpu_lib):
    p = synth.make_prefill(48, [70, 90], 8, 2, 128)
    out = _run(p, scale=0.3)
    check_rows(out, oracle.attention_prefill(p.q, p.k, p.v, p.cu_seqlens, scale=0.3), what="prefill scale")


def test_single_token_prompts_return_v_bitwise(gpu_lib):
    p = synth.make_prefill(49, [1] * 9, 16, 4, 128)
    out = _run(p)
    G = 4
    assert torch.equal(out, p.v.repeat_interleave(G, dim=1))


def test_loose_max_seqlen_and_determinism(gpu_lib):
    p = synth.make_prefill(50, [100, 33], 8, 2, 128)
    a = _run(p)
    b = _run(p, max_seqlen=133)
    assert torch.equal(a, b)


def _tile_rows(lens, first=True, last=True, tile=128):
    """Token indices of the first and/or last row of every ``tile``-row query
    block of every prompt."""
    rows, start = [], 0
    for n in lens:
        for t0 in range(0, n, tile):
            t1 = min(t0 + tile, n) - 1
            if first:
                rows.append(start + t0)
            if last:
                rows.append(start + t1)
        start += n
    return sorted(set(rows))


def test_qwen3_4096_token_prompts_every_query_tile(gpu_lib):
    """The paper's long input (two 4096-token prompts, Qwen3-32B heads): the
    first and last row of every 128-row query block of both prompts."""
    p = synth.prefill_workload("qwen3-32b", 4096, 2, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    rows = _tile_rows(pc.lens)
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens, rows=rows)
    check_rows(out[rows], ref[rows], what="qwen3-32b prefill 2x4096 (every query tile)")


def test_mixtral_128_token_prompts_all_rows(gpu_lib):
    """The paper's short input (32 prompts of 128 tokens, Mixtral heads): every row."""
    p = synth.prefill_workload("mixtral-8x7b", 128, 32, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens)
    check_rows(out, ref, what="mixtral-8x7b prefill 32x128 (all rows)")


def _cu(new):
    return torch.tensor([0] + [int(x) for x in torch.tensor(new).cumsum(0)], dtype=torch.int32)


@pytest.mark.parametrize("D,ctx,new", [
    (128, [33, 16, 7, 0, 200, 1], [33, 16, 3, 0, 190, 1]),   # prompts, full block, chunks, empty
    (64, [5, 48, 100], [5, 20, 100]),
])
def test_kv_write_bit_exact(gpu_lib, D, ctx, new):
    a = synth.custom_attention(99, len(ctx), 8, 2, D, ctx, ctx_hi=max(ctx) + 20)
    cu = _cu(new)
    T = int(cu[-1])
    kn = synth.normal_tensor(99, 42, (T, 2, D))
    vn = synth.normal_tensor(99, 43, (T, 2, D))
    rk, rv = oracle.kv_write(a.k_cache, a.v_cache, a.block_table, a.context_lens, cu, kn, vn)
    ad = a.to(DEV)
    aflex.kv_write(ad, kn.to(DEV), vn.to(DEV), cu.to(DEV), max_seqlen=max(new))
    assert torch.equal(ad.k_cache.cpu(), rk) and torch.equal(ad.v_cache.cpu(), rv)


def test_kv_write_one_token_each_matches_kv_append(gpu_lib):
    ctx = [1, 15, 16, 17, 700]
    a = synth.custom_attention(100, len(ctx), 8, 2, 128, ctx, ctx_hi=720)
    kn = synth.normal_tensor(100, 42, (len(ctx), 2, 128)).to(DEV)
    vn = synth.normal_tensor(100, 43, (len(ctx), 2, 128)).to(DEV)
    a1, a2 = a.to(DEV), a.to(DEV)
    aflex.kv_append(a1, kn, vn)
    aflex.kv_write(a2, kn, vn, torch.arange(len(ctx) + 1, dtype=torch.int32, device=DEV), max_seqlen=1)
    assert torch.equal(a1.k_cache, a2.k_cache) and torch.equal(a1.v_cache, a2.v_cache)


def test_prefill_then_decode_on_the_written_cache(gpu_lib):
    """A prefill pass writes the prompts into the paged cache; decode attention
    for each prompt's last token over that cache equals the prefill output row."""
    lens = [300, 17, 128]
    p = synth.make_prefill(101, lens, 16, 2, 128, device=DEV)
    a = synth.custom_attention(101, len(lens), 16, 2, 128, lens, ctx_hi=320).to(DEV)
    aflex.kv_write(a, p.k, p.v, p.cu_seqlens, max_seqlen=max(lens))
    out = aflex.attn_prefill(p).cpu()
    last = (p.cu_seqlens[1:] - 1).long().cpu()
    a.q = p.q[last.to(DEV)].contiguous()
    dec = aflex.attn_decode(a).cpu()
    ref = oracle.attention_prefill(p.q.cpu(), p.k.cpu(), p.v.cpu(), p.cu_seqlens.cpu(), rows=last.tolist())
    check_rows(dec, ref[last], what="decode over the prefilled cache")
    check_rows(out[last], ref[last], what="prefill last rows")


def test_long_prompt_every_query_tile(gpu_lib):
    """One 16384-token prompt at the Qwen3-32B head shape (longer than any of the
    paper's inputs): one row of every 128-row query block (its first row in
    even blocks, its last in odd ones), and the prompt's last row."""
    n = 16384
    p = synth.make_prefill(55, [n], 64, 8, 128, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    rows = sorted({t0 + (127 if (t0 // 128) % 2 else 0) for t0 in range(0, n, 128)} | {n - 1})
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens, rows=rows)
    check_rows(out[rows], ref[rows], what="prefill n=16384 (every query tile)")


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (12, 6), (64, 8)])
def test_two_heads_per_work_group_sampled(gpu_lib, Hq, Hkv):
    """Batches with a prompt of at least 2048 tokens and an even number of
    query heads per KV head run two heads per work-group: ragged long
    prompts beside a short and an empty one, sampled rows of every prompt
    (first, last, the diagonal tiles' edges); Hq / 2 not a multiple of 8 in the
    second case."""
    lens = [2048, 2100, 0, 5, 2300]
    p = synth.make_prefill(57 + Hq, lens, Hq, Hkv, 128, device=DEV)
    out = aflex.attn_prefill(p).cpu()
    pc = p.to("cpu")
    cu = [int(c) for c in pc.cu_seqlens]
    rows = []
    for b, n in enumerate(lens):
        if n:
            rows += sorted({cu[b] + r for r in (0, min(63, n - 1), min(127, n - 1), min(128, n - 1), n // 2, n - 2, n - 1) if 0 <= r < n})
    ref = oracle.attention_prefill(pc.q, pc.k, pc.v, pc.cu_seqlens, rows=rows)
    check_rows(out[rows], ref[rows], what=f"prefill two heads per work-group Hq={Hq} Hkv={Hkv} (sampled)")


def test_kv_write_long_prompt_bit_exact(gpu_lib):
    n = 5000
    a = synth.custom_attention(56, 1, 8, 8, 128, [n], ctx_hi=n)
    kn = synth.normal_tensor(56, 42, (n, 8, 128))
    vn = synth.normal_tensor(56, 43, (n, 8, 128))
    cu = torch.tensor([0, n], dtype=torch.int32)
    rk, rv = oracle.kv_write(a.k_cache, a.v_cache, a.block_table, a.context_lens, cu, kn, vn)
    ad = a.to(DEV)
    aflex.kv_write(ad, kn.to(DEV), vn.to(DEV), cu.to(DEV), max_seqlen=n)
    assert torch.equal(ad.k_cache.cpu(), rk) and torch.equal(ad.v_cache.cpu(), rv)
