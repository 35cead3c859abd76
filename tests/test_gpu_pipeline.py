"""The two-stream interleaved A/F layer step vs the oracle (through the C ABI)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _small(E=4):
    ctx = [5, 17, 40, 1, 33, 300, 9, 64]
    a = synth.custom_attention(80, 8, 4, 2, 64, ctx, ctx_hi=320)
    _, w, _ = synth.custom_ffn(80, 8, 256, 128, E=E)
    logits = torch.from_numpy(np.random.default_rng(80).standard_normal((8, max(E, 1)),
                                                                        dtype=np.float32))
    return a, w, logits


@pytest.mark.parametrize("mbs,L", [([8], 1), ([4, 4], 1), ([2, 2, 2, 2], 1), ([3, 5], 2),
                                   ([1, 1, 6], 3)])
def test_small_moe_pipeline(gpu_lib, mbs, L):
    a, w, logits = _small()
    y = aflex.af_pipeline_step(a.to(DEV), w.to(DEV), logits.to(DEV), 2, mbs, L=L).cpu()
    ref = oracle.af_layer_steps(a, w, logits, 2, mbs, L=L)
    check_rows(y, ref, what=f"pipeline mbs={mbs} L={L}")


def test_small_dense_pipeline(gpu_lib):
    a, w, _ = _small(E=0)
    y = aflex.af_pipeline_step(a.to(DEV), w.to(DEV), None, 0, [5, 3], L=2).cpu()
    check_rows(y, oracle.af_layer_steps(a, w, None, 0, [5, 3], L=2), what="dense pipeline")


def test_repeated_calls_and_explicit_streams(gpu_lib):
    a, w, logits = _small()
    ad, wd, ld = a.to(DEV), w.to(DEV), logits.to(DEV)
    sa, sf = torch.cuda.Stream(), torch.cuda.Stream()
    cur = torch.cuda.current_stream()
    sa.wait_stream(cur); sf.wait_stream(cur)
    ys = [aflex.af_pipeline_step(ad, wd, ld, 2, [2, 6], stream_a=sa, stream_f=sf) for _ in range(3)]
    cur.wait_stream(sf)
    torch.cuda.synchronize()
    assert torch.equal(ys[0], ys[1]) and torch.equal(ys[1], ys[2])


def test_af_pipeline_workload_all_rows(gpu_lib):
    """The headline workload at full size (B = 256, M = 4 microbatches of 64,
    long contexts, top-2 of 8 Mixtral experts): every row of every
    microbatch, at M = 4 and at M = 1, against the oracle's serial
    attention-then-MoE composition."""
    wl = synth.af_pipeline(device=DEV)
    a, f = wl.attn, wl.ffn
    y4 = aflex.af_pipeline_step(a, f, wl.router_logits, 2, wl.microbatches).cpu()
    y1 = aflex.af_pipeline_step(a, f, wl.router_logits, 2, [256]).cpu()
    ref = oracle.af_layer_steps(a.to("cpu"), f.to("cpu"), wl.router_logits.cpu(), 2, [256])
    check_rows(y4, ref, what="A/F pipeline M=4 (all 256 rows)")
    check_rows(y1, ref, what="A/F pipeline M=1 (all 256 rows)")


@pytest.mark.parametrize("attn_cus", [64, 128, 192])
def test_cu_pool_streams_same_result(gpu_lib, attn_cus):
    """The step on CU-partitioned streams (attention pool and FFN pool) gives the
    bitwise result of the step on ordinary streams: placement changes no
    arithmetic. The streams are released at the end, after the workspace used
    on them is freed."""
    a, w, logits = _small()
    ad, wd, ld = a.to(DEV), w.to(DEV), logits.to(DEV)
    ref = aflex.af_pipeline_step(ad, wd, ld, 2, [3, 5], L=2).clone()
    sa, sf = aflex.pool_streams(attn_cus, DEV)
    cur = torch.cuda.current_stream()
    sa.wait_stream(cur); sf.wait_stream(cur)
    ws = aflex.Workspace()
    y = aflex.af_pipeline_step(ad, wd, ld, 2, [3, 5], L=2, stream_a=sa, stream_f=sf, ws=ws)
    cur.wait_stream(sf)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    del ws
    aflex.release_pool_streams()
