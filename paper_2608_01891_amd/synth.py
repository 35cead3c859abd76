"""Seeded synthetic inputs for the decode-step Attention/FFN operators.

This module only draws inputs; it holds none of the operators' arithmetic.
Both the HIP path (through the bindings) and the CPU oracle receive what it
produces, so it depends on nothing but numpy and torch.

Two sources of randomness are used:

* Small structural draws (context lengths, the physical-block permutation,
  MoE router logits) come from numpy's PCG64 (``np.random.default_rng(seed)``)
  in a fixed order, on the host.
* Bulk bf16 tensors (q, K, V, activations, weights) come from a counter-based
  generator so that any element can be produced on any device without
  producing the ones before it. Element ``i`` of stream ``s`` takes outputs
  ``3i+1 .. 3i+3`` of SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) seeded with
  ``mix64(seed * 2**32 + s)``. Each 64-bit output is cut into four 16-bit
  uniforms and the twelve uniforms are summed (Irwin-Hall, n = 12), giving
  ``z = (sum - 393210) / 65536``, an approximately standard normal variate
  with bounded tails (|z| <= 6). All of this is integer arithmetic plus exact
  float conversions, so CPU and GPU produce identical bits. Scaled tensors
  (weights, sigma = 0.02) take one fp32 multiply; everything is rounded to
  bf16 with round-to-nearest-even.

The workloads are the decode-step operator shapes of the two models the paper
evaluates (Qwen3-32B, Mixtral-8x7B; section 6.1) at the batch sizes of its
decode characterisation (section 3) and pipeline study (section 4.3, Table 1).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

# --------------------------------------------------------------------------
# SplitMix64 in wrapping int64 torch arithmetic
# --------------------------------------------------------------------------
_MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB


def _as_i64(v: int) -> int:
    v &= _MASK64
    return v - (1 << 64) if v >= (1 << 63) else v


_GAMMA_S = _as_i64(GAMMA)
_M1_S = _as_i64(_M1)
_M2_S = _as_i64(_M2)


def _lsr(z: torch.Tensor, n: int) -> torch.Tensor:
    """Logical right shift of an int64 tensor viewed as uint64."""
    return (z >> n) & ((1 << (64 - n)) - 1)


def mix64(z: torch.Tensor) -> torch.Tensor:
    """SplitMix64 output function on int64 tensors (two's-complement wrap)."""
    z = z ^ _lsr(z, 30)
    z = z * _M1_S
    z = z ^ _lsr(z, 27)
    z = z * _M2_S
    return z ^ _lsr(z, 31)


def mix64_int(z: int) -> int:
    """The same function on Python ints (used for stream keys)."""
    z &= _MASK64
    z = ((z ^ (z >> 30)) * _M1) & _MASK64
    z = ((z ^ (z >> 27)) * _M2) & _MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, stream: int) -> int:
    return _as_i64(mix64_int(seed * (1 << 32) + stream))


def splitmix64_outputs(key: int, n: torch.Tensor) -> torch.Tensor:
    """Output number ``n`` (1-based) of SplitMix64 whose state starts at ``key``."""
    return mix64(n * _GAMMA_S + key)


def _irwin_hall12(key: int, idx: torch.Tensor) -> torch.Tensor:
    """fp32 approximately-N(0,1) variates for int64 element indices ``idx``."""
    base = idx * 3
    acc = torch.zeros_like(idx)
    for r in range(3):
        w = splitmix64_outputs(key, base + (r + 1))
        acc += (w & 0xFFFF) + ((w >> 16) & 0xFFFF) + ((w >> 32) & 0xFFFF) + ((w >> 48) & 0xFFFF)
    return (acc - 393210).to(torch.float32) * (1.0 / 65536.0)


_CHUNK = 1 << 24


def normal_at(seed: int, stream: int, idx: torch.Tensor, scale: float = 1.0,
              dtype: torch.dtype = torch.bfloat16) -> torch.Tensor:
    """Values of stream ``stream`` at the given flat indices (any device)."""
    z = _irwin_hall12(stream_key(seed, stream), idx.to(torch.int64))
    if scale != 1.0:
        z = z * torch.tensor(scale, dtype=torch.float32, device=z.device)
    return z.to(dtype)


def normal_tensor(seed: int, stream: int, shape, scale: float = 1.0,
                  device="cpu", dtype: torch.dtype = torch.bfloat16) -> torch.Tensor:
    """A whole tensor of stream ``stream``; element i of the flat view is value i."""
    numel = math.prod(shape)
    out = torch.empty(numel, dtype=dtype, device=device)
    for s in range(0, numel, _CHUNK):
        e = min(s + _CHUNK, numel)
        idx = torch.arange(s, e, dtype=torch.int64, device=device)
        out[s:e] = normal_at(seed, stream, idx, scale, dtype)
    return out.view(*shape)


# stream ids of the bulk tensors
STREAM = {"q": 1, "k": 2, "v": 3, "x": 4, "w_gate": 5, "w_up": 6, "w_down": 7,
          "prefill_q": 8, "prefill_k": 9, "prefill_v": 10,
          "k_new": 11, "v_new": 12, "w_o": 13, "x_in": 14, "norm": 15, "w_router": 16}
WEIGHT_SIGMA = 0.02
BLOCK_SIZE = 16


# --------------------------------------------------------------------------
# Structure: context lengths, block tables, router logits (numpy PCG64)
# --------------------------------------------------------------------------
def lognormal_contexts(rng: np.random.Generator, B: int, median: float, sigma: float,
                       lo: int, hi: int) -> np.ndarray:
    z = rng.standard_normal(B)
    return np.clip(np.rint(np.exp(np.log(median) + sigma * z)), lo, hi).astype(np.int32)


def paged_block_table(rng: np.random.Generator, ctx: np.ndarray, max_blocks: int,
                      block_size: int = BLOCK_SIZE):
    """Each sequence owns ceil(ctx/bs) consecutive entries of one random permutation
    of the physical blocks; unused table entries hold -1."""
    nblk = -(-ctx.astype(np.int64) // block_size)
    N = int(nblk.sum())
    perm = rng.permutation(N).astype(np.int32)
    table = np.full((len(ctx), max_blocks), -1, dtype=np.int32)
    pos = 0
    for b, n in enumerate(nblk):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    return table, N


@dataclass
class AttnInputs:
    q: torch.Tensor            # [B, Hq, D] bf16
    k_cache: torch.Tensor      # [N, Hkv, bs, D] bf16
    v_cache: torch.Tensor      # [N, Hkv, D, bs] bf16 (token index fastest)
    block_table: torch.Tensor  # [B, max_blocks] int32
    context_lens: torch.Tensor  # [B] int32
    B: int
    Hq: int
    Hkv: int
    D: int
    block_size: int
    max_blocks: int
    num_blocks: int
    max_context_len: int

    def to(self, device):
        d = dict(self.__dict__)
        for k in ("q", "k_cache", "v_cache", "block_table", "context_lens"):
            d[k] = d[k].to(device)
        return AttnInputs(**d)


@dataclass
class FFNWeights:
    w_gate: torch.Tensor   # dense [I, H]; MoE [E, I, H]
    w_up: torch.Tensor
    w_down: torch.Tensor   # dense [H, I]; MoE [E, H, I]
    H: int
    I: int
    E: int = 0

    def to(self, device):
        d = dict(self.__dict__)
        for k in ("w_gate", "w_up", "w_down"):
            d[k] = d[k].to(device)
        return FFNWeights(**d)


def make_attention(seed: int, B: int, Hq: int, Hkv: int, D: int, ctx: np.ndarray,
                   rng: np.random.Generator, ctx_hi: int, device="cpu") -> AttnInputs:
    max_blocks = -(-ctx_hi // BLOCK_SIZE)
    table, N = paged_block_table(rng, ctx, max_blocks)
    q = normal_tensor(seed, STREAM["q"], (B, Hq, D), device=device)
    k = normal_tensor(seed, STREAM["k"], (N, Hkv, BLOCK_SIZE, D), device=device)
    v = normal_tensor(seed, STREAM["v"], (N, Hkv, D, BLOCK_SIZE), device=device)
    return AttnInputs(q=q, k_cache=k, v_cache=v,
                      block_table=torch.from_numpy(table).to(device),
                      context_lens=torch.from_numpy(ctx.astype(np.int32)).to(device),
                      B=B, Hq=Hq, Hkv=Hkv, D=D, block_size=BLOCK_SIZE,
                      max_blocks=max_blocks, num_blocks=N,
                      max_context_len=int(max_blocks * BLOCK_SIZE))


def make_ffn_weights(seed: int, H: int, I: int, E: int = 0, device="cpu") -> FFNWeights:
    lead = (E,) if E else ()
    wg = normal_tensor(seed, STREAM["w_gate"], lead + (I, H), WEIGHT_SIGMA, device)
    wu = normal_tensor(seed, STREAM["w_up"], lead + (I, H), WEIGHT_SIGMA, device)
    wd = normal_tensor(seed, STREAM["w_down"], lead + (H, I), WEIGHT_SIGMA, device)
    return FFNWeights(w_gate=wg, w_up=wu, w_down=wd, H=H, I=I, E=E)


# --------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    seed: int
    attn: AttnInputs | None = None
    x: torch.Tensor | None = None          # [T, H] bf16 FFN input
    ffn: FFNWeights | None = None
    router_logits: torch.Tensor | None = None  # [T, E] fp32
    top_k: int = 0
    microbatches: list = field(default_factory=list)
    meta: dict = field(default_factory=dict)


def tiny_layer(device="cpu") -> Workload:
    """Tiny decoder layer: B=4, 8/2 heads, D=64, ctx ~ U[17,200], SwiGLU 512->1408."""
    seed = 0
    rng = np.random.default_rng(seed)
    ctx = rng.integers(17, 201, 4).astype(np.int32)
    attn = make_attention(seed, 4, 8, 2, 64, ctx, rng, ctx_hi=200, device=device)
    x = normal_tensor(seed, STREAM["x"], (4, 512), device=device)
    ffn = make_ffn_weights(seed, 512, 1408, device=device)
    return Workload("tiny-layer", seed, attn=attn, x=x, ffn=ffn)


def qwen3_attention(device="cpu") -> Workload:
    """Qwen3-32B decode attention: B=64, 64/8 heads, D=128, lognormal ctx."""
    seed = 1
    rng = np.random.default_rng(seed)
    ctx = lognormal_contexts(rng, 64, 1024, 0.8, 64, 8192)
    attn = make_attention(seed, 64, 64, 8, 128, ctx, rng, ctx_hi=8192, device=device)
    return Workload("qwen3-32b-decode-attention", seed, attn=attn)


def qwen3_swiglu(T: int, device="cpu", weights: FFNWeights | None = None) -> Workload:
    """Qwen3-32B dense SwiGLU: H=5120, I=25600; x is the first T rows of a 512-row draw."""
    seed = 2
    assert 1 <= T <= 512
    ffn = weights if weights is not None else make_ffn_weights(seed, 5120, 25600, device=device)
    x = normal_tensor(seed, STREAM["x"], (512, 5120), device=device)[:T].contiguous()
    return Workload(f"qwen3-32b-swiglu-T{T}", seed, x=x, ffn=ffn, meta={"T": T})


def mixtral_moe(device="cpu", T: int = 256, seed: int = 3,
                weights: FFNWeights | None = None) -> Workload:
    """Mixtral-8x7B MoE: H=4096, 8 experts of I=14336, top-2, T tokens."""
    rng = np.random.default_rng(seed)
    logits = rng.standard_normal((T, 8), dtype=np.float32)
    x = normal_tensor(seed, STREAM["x"], (T, 4096), device=device)
    ffn = weights if weights is not None else make_ffn_weights(seed, 4096, 14336, E=8, device=device)
    return Workload(f"mixtral-8x7b-moe-T{T}", seed, x=x, ffn=ffn,
                    router_logits=torch.from_numpy(logits).to(device), top_k=2)


def af_pipeline(device="cpu", M: int = 4) -> Workload:
    """Interleaved A/F layer step: B=256, 32/8 heads, D=128, long lognormal ctx,
    Mixtral top-2 MoE FFN on each of M microbatches."""
    seed = 4
    rng = np.random.default_rng(seed)
    ctx = lognormal_contexts(rng, 256, 4096, 0.7, 256, 32768)
    attn = make_attention(seed, 256, 32, 8, 128, ctx, rng, ctx_hi=32768, device=device)
    logits = rng.standard_normal((256, 8), dtype=np.float32)
    ffn = make_ffn_weights(seed, 4096, 14336, E=8, device=device)
    mbs = [256 // M] * M
    return Workload(f"af-pipeline-B256-M{M}", seed, attn=attn, ffn=ffn,
                    router_logits=torch.from_numpy(logits).to(device), top_k=2,
                    microbatches=mbs)


@dataclass
class PrefillInputs:
    q: torch.Tensor           # [T, Hq, D] bf16, prompts packed back to back
    k: torch.Tensor           # [T, Hkv, D] bf16
    v: torch.Tensor           # [T, Hkv, D] bf16
    cu_seqlens: torch.Tensor  # [B + 1] int32, prompt b is tokens cu[b] .. cu[b+1] - 1
    lens: list
    Hq: int
    Hkv: int
    D: int

    @property
    def T(self) -> int:
        return int(sum(self.lens))

    @property
    def max_seqlen(self) -> int:
        return max(max(self.lens), 0)

    def to(self, device):
        d = dict(self.__dict__)
        for k in ("q", "k", "v", "cu_seqlens"):
            d[k] = d[k].to(device)
        return PrefillInputs(**d)


def make_prefill(seed: int, lens, Hq: int, Hkv: int, D: int, device="cpu") -> PrefillInputs:
    """Packed prompts of the given lengths; q, k, v are standard normal bf16."""
    lens = [int(n) for n in lens]
    cu = np.concatenate([[0], np.cumsum(lens, dtype=np.int64)]).astype(np.int32)
    T = int(cu[-1])
    q = normal_tensor(seed, STREAM["prefill_q"], (T, Hq, D), device=device)
    k = normal_tensor(seed, STREAM["prefill_k"], (T, Hkv, D), device=device)
    v = normal_tensor(seed, STREAM["prefill_v"], (T, Hkv, D), device=device)
    return PrefillInputs(q=q, k=k, v=v, cu_seqlens=torch.from_numpy(cu).to(device),
                         lens=lens, Hq=Hq, Hkv=Hkv, D=D)


# Prefill workloads at the paper's two prompt lengths (section 6.1: 128- and
# 4096-token inputs), with the attention shapes of the two models.
PREFILL_SHAPES = {"qwen3-32b": (64, 8, 128), "mixtral-8x7b": (32, 8, 128)}


def prefill_workload(model: str = "qwen3-32b", prompt_len: int = 4096, prompts: int = 2,
                     device="cpu") -> PrefillInputs:
    Hq, Hkv, D = PREFILL_SHAPES[model]
    seed = 5 if prompt_len >= 1024 else 6
    return make_prefill(seed, [prompt_len] * prompts, Hq, Hkv, D, device=device)


def prefill_ffn_tokens(H: int, T: int, device="cpu") -> torch.Tensor:
    """FFN input [T, H] of a prefill batch (all prompt tokens at once)."""
    return normal_tensor(7, STREAM["x"], (T, H), device=device)


@dataclass
class LayerInputs:
    """The rest of a decode layer around the A/F operator pair: the new token's
    K/V per sequence, the output projection, the layer input (residual) and the
    MoE block's RMSNorm gain and router."""
    k_new: torch.Tensor          # [B, Hkv, D] bf16
    v_new: torch.Tensor          # [B, Hkv, D] bf16
    w_o: torch.Tensor            # [H, Hq * D] bf16
    x_in: torch.Tensor | None    # [B, H] bf16 (None: no residual on the projection)
    norm_weight: torch.Tensor    # [H] bf16
    router_weight: torch.Tensor  # [E, H] bf16
    eps: float = 1e-5

    def to(self, device):
        d = dict(self.__dict__)
        for k in ("k_new", "v_new", "w_o", "x_in", "norm_weight", "router_weight"):
            if d[k] is not None:
                d[k] = d[k].to(device)
        return LayerInputs(**d)


def make_layer(seed: int, B: int, Hq: int, Hkv: int, D: int, H: int, E: int, residual: bool = True,
               device="cpu") -> LayerInputs:
    """Decode-layer inputs: K/V and x ~ N(0,1), W_o and W_r ~ N(0, 0.02),
    RMSNorm gain 1 + 0.1 N(0,1) (all bf16)."""
    kn = normal_tensor(seed, STREAM["k_new"], (B, Hkv, D), device=device)
    vn = normal_tensor(seed, STREAM["v_new"], (B, Hkv, D), device=device)
    wo = normal_tensor(seed, STREAM["w_o"], (H, Hq * D), WEIGHT_SIGMA, device)
    x = normal_tensor(seed, STREAM["x_in"], (B, H), device=device) if residual else None
    g = (1.0 + 0.1 * normal_tensor(seed, STREAM["norm"], (H,), dtype=torch.float32, device=device)
         ).to(torch.bfloat16)
    wr = normal_tensor(seed, STREAM["w_router"], (E, H), WEIGHT_SIGMA, device)
    return LayerInputs(k_new=kn, v_new=vn, w_o=wo, x_in=x, norm_weight=g, router_weight=wr)


def custom_attention(seed: int, B: int, Hq: int, Hkv: int, D: int, ctx, ctx_hi: int | None = None,
                     device="cpu") -> AttnInputs:
    """Attention inputs with given context lengths (tests: edge cases, ragged tails)."""
    rng = np.random.default_rng(seed)
    ctx = np.asarray(ctx, dtype=np.int32)
    hi = int(ctx_hi if ctx_hi is not None else max(int(ctx.max()), 1))
    return make_attention(seed, B, Hq, Hkv, D, ctx, rng, ctx_hi=hi, device=device)


def custom_ffn(seed: int, T: int, H: int, I: int, E: int = 0, device="cpu"):
    """FFN / MoE inputs of arbitrary shape (tests)."""
    rng = np.random.default_rng(seed)
    logits = rng.standard_normal((T, max(E, 1)), dtype=np.float32)
    x = normal_tensor(seed, STREAM["x"], (T, H), device=device)
    w = make_ffn_weights(seed, H, I, E, device=device)
    return x, w, torch.from_numpy(logits).to(device)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a CPU bf16 tensor as uint16."""
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)
