"""HIP dense SwiGLU FFN vs the oracle (through the C ABI)."""
import pytest
import torch

import oracle
from paper_2608_01891_amd import aflex, synth
from tests.helpers import sample_rows
from tests.parity import check_rows

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_tiny_layer(gpu_lib):
    w = synth.tiny_layer()
    y = aflex.ffn_swiglu(w.x.to(DEV), w.ffn.to(DEV)).cpu()
    check_rows(y, oracle.swiglu_ffn(w.x, w.ffn.w_gate, w.ffn.w_up, w.ffn.w_down), what="tiny swiglu")


@pytest.mark.parametrize("T,H,I", [(1, 256, 320), (33, 320, 192), (200, 192, 448), (130, 640, 1408)])
def test_ragged_shapes(gpu_lib, T, H, I):
    x, w, _ = synth.custom_ffn(50 + T, T, H, I)
    y = aflex.ffn_swiglu(x.to(DEV), w.to(DEV)).cpu()
    check_rows(y, oracle.swiglu_ffn(x, w.w_gate, w.w_up, w.w_down), what=f"swiglu T={T} H={H} I={I}")


@pytest.fixture(scope="module")
def qwen3_weights():
    w = synth.make_ffn_weights(2, 5120, 25600, device=DEV)
    cpu64 = (w.w_gate.cpu().double(), w.w_up.cpu().double(), w.w_down.cpu().double())
    yield w, cpu64
    del w


@pytest.mark.parametrize("T", [32, 128, 256, 512])
def test_qwen3_shape_all_rows(gpu_lib, qwen3_weights, T):
    """Qwen3-32B SwiGLU at every decode batch of the workload, every row."""
    w, (wg, wu, wd) = qwen3_weights
    wl = synth.qwen3_swiglu(T, device=DEV, weights=w)
    y = aflex.ffn_swiglu(wl.x, w).cpu()
    ref = oracle.swiglu_ffn(wl.x.cpu(), wg, wu, wd)
    check_rows(y, ref, what=f"qwen3 swiglu T={T} (all rows)")
    y2 = aflex.ffn_swiglu(wl.x, w).cpu()
    assert torch.equal(y, y2)


def test_qwen3_prefill_tokens_every_row_tile(gpu_lib, qwen3_weights):
    """The dense FFN over a prefill batch: two 2048-token prompts at once
    (T = 4096), the first and last row of every 256-row block plus random
    rows."""
    w, (wg, wu, wd) = qwen3_weights
    T = 4096
    x = synth.prefill_ffn_tokens(5120, T, device=DEV)
    y = aflex.ffn_swiglu(x, w).cpu()
    edges = [r for t0 in range(0, T, 256) for r in (t0, t0 + 255)]
    rows = sample_rows(T, len(edges) + 8, seed=T, must=edges)
    ref = oracle.swiglu_ffn(x[rows].cpu(), wg, wu, wd)
    check_rows(y[rows], ref, what="qwen3 swiglu prefill T=4096 (every 256-row block)")


@pytest.mark.parametrize("T", [32, 33, 64, 65, 100, 255, 257, 300, 406, 456, 511])
def test_tile_plan_boundaries(gpu_lib, T):
    """Token counts on both sides of the dense tile-size thresholds, and
    partly filled last row tiles whose waves multiply 0 to 4 of their row
    blocks (128-row tile with 100 rows; 256-row tails of 1, 44, 150, 200 and
    255 rows)."""
    x, w, _ = synth.custom_ffn(120 + T, T, 320, 640)
    y = aflex.ffn_swiglu(x.to(DEV), w.to(DEV)).cpu()
    check_rows(y, oracle.swiglu_ffn(x, w.w_gate, w.w_up, w.w_down), what=f"swiglu T={T}")


@pytest.mark.parametrize("T,H,I", [(8, 128, 7168), (20, 128, 5120)])
def test_many_down_splits(gpu_lib, T, H, I):
    """A narrow output and a wide intermediate size split the down GEMM into
    14 and 10 K slices, which the reduce sums in batches of four (the last
    batch partly used)."""
    x, w, _ = synth.custom_ffn(130 + T, T, H, I)
    y = aflex.ffn_swiglu(x.to(DEV), w.to(DEV)).cpu()
    check_rows(y, oracle.swiglu_ffn(x, w.w_gate, w.w_up, w.w_down), what=f"swiglu many splits T={T} I={I}")
