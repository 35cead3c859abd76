"""The seeded input generator: published SplitMix64 values, device-independent
bits, distribution moments and the structural check values of the workloads."""
import random

import numpy as np
import pytest
import torch

from paper_2608_01891_amd import synth


def _splitmix64_reference(seed, n):
    """Pure-Python SplitMix64 written from its published definition."""
    out, x = [], seed
    for _ in range(n):
        x = (x + 0x9E3779B97F4A7C15) & ((1 << 64) - 1)
        z = x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & ((1 << 64) - 1)
        out.append(z ^ (z >> 31))
    return out


def test_splitmix64_published_first_outputs():
    # the first three outputs of SplitMix64 seeded with 0
    assert _splitmix64_reference(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4,
                                           0x06C45D188009454F]


def test_torch_splitmix64_matches_reference():
    rnd = random.Random(7)
    for _ in range(20):
        seed = rnd.getrandbits(64)
        ref = _splitmix64_reference(seed, 64)
        key = synth._as_i64(seed)
        got = synth.splitmix64_outputs(key, torch.arange(1, 65, dtype=torch.int64))
        assert [v & ((1 << 64) - 1) for v in got.tolist()] == ref


def test_normal_at_matches_whole_tensor_and_is_deterministic():
    t = synth.normal_tensor(5, 3, (1000,), scale=0.02)
    idx = torch.tensor([0, 17, 999, 512])
    assert torch.equal(synth.normal_at(5, 3, idx, scale=0.02), t[idx])
    assert torch.equal(t, synth.normal_tensor(5, 3, (1000,), scale=0.02))
    assert not torch.equal(t, synth.normal_tensor(5, 4, (1000,), scale=0.02))


def test_irwin_hall_moments():
    z = synth.normal_tensor(11, 1, (1 << 20,), dtype=torch.float32).double()
    assert abs(z.mean()) < 5e-3
    assert abs(z.var() - 1.0) < 5e-3
    assert z.abs().max() <= 6.0
    # excess kurtosis of Irwin-Hall(12) is -0.1
    k = ((z - z.mean()) ** 4).mean() / z.var() ** 2 - 3.0
    assert -0.2 < float(k) < 0.0


def test_tiny_layer_structure():
    w = synth.tiny_layer()
    assert w.attn.context_lens.tolist() == [173, 134, 111, 66]
    assert w.attn.num_blocks == 32
    bt = w.attn.block_table
    used = bt[bt >= 0]
    assert sorted(used.tolist()) == list(range(32))
    for b, c in enumerate(w.attn.context_lens.tolist()):
        n = -(-c // 16)
        assert (bt[b, :n] >= 0).all() and (bt[b, n:] == -1).all()


def test_workload_check_values():
    rng = np.random.default_rng(1)
    ctx = synth.lognormal_contexts(rng, 64, 1024, 0.8, 64, 8192)
    assert (int(ctx.sum()), int(ctx.min()), int(ctx.max())) == (77755, 117, 5573)
    assert int((-(-ctx // 16)).sum()) == 4893
    rng = np.random.default_rng(4)
    ctx = synth.lognormal_contexts(rng, 256, 4096, 0.7, 256, 32768)
    assert (int(ctx.sum()), int(ctx.min()), int(ctx.max())) == (1392790, 511, 22384)
    assert [int(ctx[i * 64:(i + 1) * 64].sum()) for i in range(4)] == [321783, 367282, 341171,
                                                                      362554]
    assert int((-(-ctx // 16)).sum()) == 87176


def test_bf16_bits_roundtrip():
    t = synth.normal_tensor(0, 1, (64,))
    bits = synth.bf16_bits(t)
    back = torch.from_numpy((bits.astype(np.uint32) << 16).view(np.float32))
    assert torch.equal(back, t.float())
