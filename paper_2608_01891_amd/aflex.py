"""Python binding of libaflex.so (ctypes; argument marshalling only).

Every computation runs in the library's HIP kernels; this module only turns
torch device tensors into pointers and sizes, sizes the workspace, and maps
status codes to exceptions. It never falls back to another implementation:
if the library is not built or no GPU is present, calls raise.
"""
from __future__ import annotations

import atexit
import ctypes
import gc
import os
import re

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libaflex.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "aflex.h")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_ALIGNMENT, ERR_WORKSPACE, ERR_HIP = range(6)

_p = ctypes.c_void_p
_i = ctypes.c_int32


class AttnArgs(ctypes.Structure):
    _fields_ = [("q", _p), ("k_cache", _p), ("v_cache", _p), ("block_table", _p),
                ("context_lens", _p), ("out", _p),
                ("B", _i), ("Hq", _i), ("Hkv", _i), ("D", _i), ("block_size", _i),
                ("max_blocks_per_seq", _i), ("num_blocks", _i), ("max_context_len", _i),
                ("scale", ctypes.c_float), ("split_tokens", _i)]


class FfnArgs(ctypes.Structure):
    _fields_ = [("x", _p), ("router_logits", _p), ("w_gate", _p), ("w_up", _p), ("w_down", _p),
                ("y", _p), ("topk_ids", _p), ("topk_w", _p), ("expert_offsets", _p),
                ("sorted_pairs", _p),
                ("T", _i), ("H", _i), ("I", _i), ("E", _i), ("k", _i)]


class KvAppendArgs(ctypes.Structure):
    _fields_ = [("k_new", _p), ("v_new", _p), ("k_cache", _p), ("v_cache", _p),
                ("block_table", _p), ("context_lens", _p),
                ("B", _i), ("Hkv", _i), ("D", _i), ("block_size", _i),
                ("max_blocks_per_seq", _i), ("num_blocks", _i)]


class LinearArgs(ctypes.Structure):
    _fields_ = [("x", _p), ("w", _p), ("y", _p), ("T", _i), ("K", _i), ("N", _i)]


class MoeBlockArgs(ctypes.Structure):
    _fields_ = [("ffn", FfnArgs), ("norm_weight", _p), ("router_weight", _p),
                ("eps", ctypes.c_float), ("residual", _i), ("router_logits_out", _p)]


class KvWriteArgs(ctypes.Structure):
    _fields_ = [("k_new", _p), ("v_new", _p), ("cu_seqlens", _p), ("k_cache", _p), ("v_cache", _p),
                ("block_table", _p), ("context_lens", _p),
                ("B", _i), ("T", _i), ("Hkv", _i), ("D", _i), ("max_seqlen", _i), ("block_size", _i),
                ("max_blocks_per_seq", _i), ("num_blocks", _i)]


class PrefillArgs(ctypes.Structure):
    _fields_ = [("q", _p), ("k", _p), ("v", _p), ("cu_seqlens", _p), ("out", _p),
                ("B", _i), ("T", _i), ("Hq", _i), ("Hkv", _i), ("D", _i),
                ("max_seqlen", _i), ("scale", ctypes.c_float)]


class LayerArgs(ctypes.Structure):
    _fields_ = [("k_new", _p), ("v_new", _p), ("k_cache", _p), ("v_cache", _p), ("w_o", _p),
                ("x_in", _p), ("norm_weight", _p), ("router_weight", _p), ("eps", ctypes.c_float)]


class AflexError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"aflex status {status}: {message}")
        self.status = status


_lib = None
_SZ = ctypes.POINTER(ctypes.c_size_t)


def exported_names():
    """Function names declared in include/aflex.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(aflex_\w+)\s*\(", text, re.M)))


def load():
    """Open the built library (cached). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_01891_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    AP, FP = ctypes.POINTER(AttnArgs), ctypes.POINTER(FfnArgs)
    I32P = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "aflex_attn_decode_workspace": [AP, _SZ],
        "aflex_attn_decode": [AP, _p, ctypes.c_size_t, _p],
        "aflex_attn_decode_noalloc": [AP, _p],
        "aflex_ffn_swiglu_workspace": [FP, _SZ],
        "aflex_ffn_swiglu": [FP, _p, ctypes.c_size_t, _p],
        "aflex_moe_ffn_workspace": [FP, _SZ],
        "aflex_moe_ffn": [FP, _p, ctypes.c_size_t, _p],
        "aflex_af_pipeline_workspace": [AP, FP, _i, I32P, _i, _SZ],
        "aflex_af_pipeline_step": [AP, FP, _i, I32P, _i, _p, ctypes.c_size_t, _p, _p],
        "aflex_af_layer_workspace": [AP, FP, ctypes.POINTER(LayerArgs), _i, I32P, _i, _SZ],
        "aflex_af_layer_step": [AP, FP, ctypes.POINTER(LayerArgs), _i, I32P, _i, _p, ctypes.c_size_t, _p, _p],
        "aflex_kv_append": [ctypes.POINTER(KvAppendArgs), _p],
        "aflex_moe_block_workspace": [ctypes.POINTER(MoeBlockArgs), _SZ],
        "aflex_moe_block": [ctypes.POINTER(MoeBlockArgs), _p, ctypes.c_size_t, _p],
        "aflex_linear_workspace": [ctypes.POINTER(LinearArgs), _SZ],
        "aflex_linear": [ctypes.POINTER(LinearArgs), _p, ctypes.c_size_t, _p],
        "aflex_attn_prefill": [ctypes.POINTER(PrefillArgs), _p],
        "aflex_kv_write": [ctypes.POINTER(KvWriteArgs), _p],
        "aflex_pool_streams_create": [ctypes.c_int32, ctypes.POINTER(_p), ctypes.POINTER(_p)],
        "aflex_pool_streams_destroy": [_p, _p],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.aflex_profile_start.argtypes = [ctypes.c_char_p]
    lib.aflex_profile_start.restype = ctypes.c_int
    lib.aflex_profile_stop.argtypes = [ctypes.c_char_p, ctypes.c_size_t]
    lib.aflex_profile_stop.restype = ctypes.c_int
    lib.aflex_teardown.argtypes = []
    lib.aflex_teardown.restype = ctypes.c_int
    lib.aflex_last_error.restype = ctypes.c_char_p
    lib.aflex_version.restype = ctypes.c_char_p
    _lib = lib
    atexit.register(close)
    return lib


def release_pool_streams():
    """Destroy the CU-partitioned stream pairs created by pool_streams().

    torch records an event on every stream a tensor was used on (record_stream)
    when that tensor is freed, so such tensors must go first: this drops the
    binding's own default workspaces (which record the streams they are used
    on), waits for the devices and lets torch retire those events, then
    destroys the streams. Buffers the caller used on the pool streams with
    record_stream must be freed before the call."""
    if not _pool_streams:
        return
    _default_ws.clear()
    gc.collect()
    for d in {key[0] for key in _pool_streams}:
        torch.cuda.synchronize(d)
    torch.cuda.empty_cache()
    first = OK
    for key in list(_pool_streams):
        sa, sf = _pool_streams.pop(key)
        st = _lib.aflex_pool_streams_destroy(_p(sa.cuda_stream), _p(sf.cuda_stream))
        first = st if first == OK else first
    _check(first)


def close():
    """Release what the library and this binding hold on the GPU: the pool
    streams (release_pool_streams) and, once the devices are idle, the
    library's cached HIP events (aflex_teardown). Registered to run at
    interpreter exit, so that no HIP object of ours is left for the runtime's
    own teardown; the library stays usable afterwards (a later call re-creates
    what it needs)."""
    if _lib is None:
        return
    release_pool_streams()
    if torch.cuda.is_initialized():
        for d in range(torch.cuda.device_count()):
            torch.cuda.synchronize(d)
    _check(_lib.aflex_teardown())


def profile_start(kernels=None):
    """Start per-kernel event timing for the named library kernels (None = all)."""
    lib = load()
    _check(lib.aflex_profile_start(",".join(kernels).encode() if kernels else None))


def profile_stop():
    """Stop timing; {kernel: (launches, total_ms, min_ms, max_ms)}."""
    lib = load()
    buf = ctypes.create_string_buffer(1 << 16)
    _check(lib.aflex_profile_stop(buf, len(buf)))
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, tot, mn, mx = line.split()
        out[name] = (int(n), float(tot), float(mn), float(mx))
    return out


def _check(status: int):
    if status != OK:
        raise AflexError(status, _lib.aflex_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(s):
    if s is None:
        s = torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Workspace:
    """Grow-only device scratch handed to the library (allocated by torch)."""

    def __init__(self, device=None):
        self.device = device
        self.buf = None

    def get(self, nbytes: int, device):
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != torch.device(device):
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        return self.buf


_default_ws = {}


def _ws(key, nbytes, device, ws, streams=()):
    """Workspace pointer and size. The buffer comes from torch's caching allocator
    on the current stream; its use on any other stream is recorded, so that a
    later growth (which frees it) cannot hand the memory out while that stream
    still reads it."""
    if ws is None:
        ws = _default_ws.setdefault(key, Workspace())
    buf = ws.get(nbytes, device)
    cur = torch.cuda.current_stream(buf.device)
    for s in streams:
        if s is not None and s != cur:
            buf.record_stream(s)
    return ctypes.c_void_p(buf.data_ptr()), ctypes.c_size_t(buf.numel())


# --------------------------------------------------------------------------
def attn_args(a, out=None, split_tokens: int = 0, scale: float = 0.0) -> AttnArgs:
    """Argument block from synth.AttnInputs-like attributes (device tensors)."""
    return AttnArgs(q=_ptr(a.q), k_cache=_ptr(a.k_cache), v_cache=_ptr(a.v_cache),
                    block_table=_ptr(a.block_table), context_lens=_ptr(a.context_lens),
                    out=_ptr(out), B=a.B, Hq=a.Hq, Hkv=a.Hkv, D=a.D, block_size=a.block_size,
                    max_blocks_per_seq=a.max_blocks, num_blocks=a.num_blocks,
                    max_context_len=a.max_context_len, scale=scale, split_tokens=split_tokens)


def ffn_args(x, w, y, logits=None, k: int = 0, routing=None) -> FfnArgs:
    T = (x.shape[0] if x is not None else y.shape[0])
    r = routing or {}
    return FfnArgs(x=_ptr(x), router_logits=_ptr(logits), w_gate=_ptr(w.w_gate),
                   w_up=_ptr(w.w_up), w_down=_ptr(w.w_down), y=_ptr(y),
                   topk_ids=_ptr(r.get("topk_ids")), topk_w=_ptr(r.get("topk_w")),
                   expert_offsets=_ptr(r.get("expert_offsets")),
                   sorted_pairs=_ptr(r.get("sorted_pairs")),
                   T=T, H=w.H, I=w.I, E=w.E, k=k)


def attn_decode(a, out=None, split_tokens: int = 0, scale: float = 0.0, stream=None, ws=None):
    lib = load()
    if out is None:
        out = torch.empty(a.B, a.Hq, a.D, dtype=torch.bfloat16, device=a.q.device)
    args = attn_args(a, out, split_tokens, scale)
    n = ctypes.c_size_t()
    _check(lib.aflex_attn_decode_workspace(ctypes.byref(args), ctypes.byref(n)))
    p, sz = _ws("attn", n.value, a.q.device, ws, (stream,))
    _check(lib.aflex_attn_decode(ctypes.byref(args), p, sz, _stream(stream)))
    return out


def attn_decode_noalloc(a, out, split_tokens: int = 0, scale: float = 0.0, stream=None):
    """Decode attention into ``out`` without a workspace: the library's static
    device scratch holds the split partials (calls on one device must not
    overlap)."""
    lib = load()
    args = attn_args(a, out, split_tokens, scale)
    _check(lib.aflex_attn_decode_noalloc(ctypes.byref(args), _stream(stream)))
    return out


def ffn_swiglu(x, w, y=None, stream=None, ws=None):
    lib = load()
    if y is None:
        y = torch.empty(x.shape[0], w.H, dtype=torch.bfloat16, device=x.device)
    args = ffn_args(x, w, y)
    n = ctypes.c_size_t()
    _check(lib.aflex_ffn_swiglu_workspace(ctypes.byref(args), ctypes.byref(n)))
    p, sz = _ws("ffn", n.value, x.device, ws, (stream,))
    _check(lib.aflex_ffn_swiglu(ctypes.byref(args), p, sz, _stream(stream)))
    return y


def moe_ffn(x, w, logits, k: int, y=None, routing: bool = False, stream=None, ws=None):
    """y [T, H]; with routing=True also the topk ids/weights, offsets and pair order."""
    lib = load()
    T = x.shape[0]
    if y is None:
        y = torch.empty(T, w.H, dtype=torch.bfloat16, device=x.device)
    r = None
    if routing:
        r = {"topk_ids": torch.empty(T, k, dtype=torch.int32, device=x.device),
             "topk_w": torch.empty(T, k, dtype=torch.float32, device=x.device),
             "expert_offsets": torch.empty(w.E + 1, dtype=torch.int32, device=x.device),
             "sorted_pairs": torch.empty(T * k, dtype=torch.int32, device=x.device)}
    args = ffn_args(x, w, y, logits, k, r)
    n = ctypes.c_size_t()
    _check(lib.aflex_moe_ffn_workspace(ctypes.byref(args), ctypes.byref(n)))
    p, sz = _ws("moe", n.value, x.device, ws, (stream,))
    _check(lib.aflex_moe_ffn(ctypes.byref(args), p, sz, _stream(stream)))
    return (y, r) if routing else y


def kv_append(a, k_new, v_new, stream=None):
    """Write each sequence's new token (position ctx-1) into a's paged pools, in place."""
    lib = load()
    args = KvAppendArgs(k_new=_ptr(k_new), v_new=_ptr(v_new), k_cache=_ptr(a.k_cache),
                        v_cache=_ptr(a.v_cache), block_table=_ptr(a.block_table),
                        context_lens=_ptr(a.context_lens), B=a.B, Hkv=a.Hkv, D=a.D,
                        block_size=a.block_size, max_blocks_per_seq=a.max_blocks,
                        num_blocks=a.num_blocks)
    _check(lib.aflex_kv_append(ctypes.byref(args), _stream(stream)))


def kv_write(a, k_new, v_new, cu_seqlens, max_seqlen=None, stream=None):
    """Write packed new tokens (rows cu[b] .. cu[b+1]-1 for sequence b) at the end of each
    sequence's context in a's paged pools, in place."""
    lib = load()
    T = k_new.shape[0]
    if max_seqlen is None:
        c = cu_seqlens.cpu()
        max_seqlen = int((c[1:] - c[:-1]).max()) if c.numel() > 1 else 0
    args = KvWriteArgs(k_new=_ptr(k_new), v_new=_ptr(v_new), cu_seqlens=_ptr(cu_seqlens),
                       k_cache=_ptr(a.k_cache), v_cache=_ptr(a.v_cache), block_table=_ptr(a.block_table),
                       context_lens=_ptr(a.context_lens), B=a.B, T=T, Hkv=a.Hkv, D=a.D,
                       max_seqlen=max_seqlen, block_size=a.block_size, max_blocks_per_seq=a.max_blocks,
                       num_blocks=a.num_blocks)
    _check(lib.aflex_kv_write(ctypes.byref(args), _stream(stream)))


def attn_prefill(p, out=None, max_seqlen=None, scale: float = 0.0, stream=None):
    """Causal attention over the packed prompts of ``p`` (synth.PrefillInputs on the device)."""
    lib = load()
    T, Hq, D = p.q.shape
    if out is None:
        out = torch.empty(T, Hq, D, dtype=torch.bfloat16, device=p.q.device)
    args = PrefillArgs(q=_ptr(p.q), k=_ptr(p.k), v=_ptr(p.v), cu_seqlens=_ptr(p.cu_seqlens),
                       out=_ptr(out), B=p.cu_seqlens.numel() - 1, T=T, Hq=Hq, Hkv=p.k.shape[1], D=D,
                       max_seqlen=p.max_seqlen if max_seqlen is None else max_seqlen, scale=scale)
    _check(lib.aflex_attn_prefill(ctypes.byref(args), _stream(stream)))
    return out


def linear(x, w, y=None, stream=None, ws=None):
    """y = x w^T (bf16), x [T, K], w [N, K]."""
    lib = load()
    T, K = x.shape
    N = w.shape[0]
    if y is None:
        y = torch.empty(T, N, dtype=torch.bfloat16, device=x.device)
    args = LinearArgs(x=_ptr(x), w=_ptr(w), y=_ptr(y), T=T, K=K, N=N)
    n = ctypes.c_size_t()
    _check(lib.aflex_linear_workspace(ctypes.byref(args), ctypes.byref(n)))
    p, sz = _ws("linear", n.value, x.device, ws, (stream,))
    _check(lib.aflex_linear(ctypes.byref(args), p, sz, _stream(stream)))
    return y


def moe_block(x, w, norm_weight, router_weight, k: int, eps: float = 1e-5, residual: bool = False,
              y=None, routing: bool = False, stream=None, ws=None):
    """y = MoE(RMSNorm(x)) (+ x): normalisation, router GEMM and experts on the device.

    With routing=True also returns the router logits and the routing outputs."""
    lib = load()
    T = x.shape[0]
    if y is None:
        y = torch.empty(T, w.H, dtype=torch.bfloat16, device=x.device)
    r = None
    logits = None
    if routing:
        r = {"topk_ids": torch.empty(T, k, dtype=torch.int32, device=x.device),
             "topk_w": torch.empty(T, k, dtype=torch.float32, device=x.device),
             "expert_offsets": torch.empty(w.E + 1, dtype=torch.int32, device=x.device),
             "sorted_pairs": torch.empty(T * k, dtype=torch.int32, device=x.device)}
        logits = torch.empty(T, w.E, dtype=torch.float32, device=x.device)
    args = MoeBlockArgs(ffn=ffn_args(x, w, y, None, k, r), norm_weight=_ptr(norm_weight),
                        router_weight=_ptr(router_weight), eps=eps, residual=int(residual),
                        router_logits_out=_ptr(logits))
    n = ctypes.c_size_t()
    _check(lib.aflex_moe_block_workspace(ctypes.byref(args), ctypes.byref(n)))
    p, sz = _ws("moe_block", n.value, x.device, ws, (stream,))
    _check(lib.aflex_moe_block(ctypes.byref(args), p, sz, _stream(stream)))
    return (y, logits, r) if routing else y


_pipe_streams = {}


def pipeline_streams(device):
    """A pair of default-priority side streams for the two pipeline stages."""
    d = torch.device(device)
    if d not in _pipe_streams:
        _pipe_streams[d] = (torch.cuda.Stream(device=d), torch.cuda.Stream(device=d))
    return _pipe_streams[d]


_pool_streams = {}


def pool_streams(attn_cus: int, device="cuda:0"):
    """Stream pair on disjoint CU sets (attn_cus of 256 CUs for the attention stage),
    as torch external streams; created once per (device, attn_cus) and destroyed
    by release_pool_streams() (by close() at interpreter exit at the latest)."""
    d = torch.device(device)
    key = (d, attn_cus)
    if key not in _pool_streams:
        lib = load()
        with torch.cuda.device(d):
            sa, sf = _p(), _p()
            _check(lib.aflex_pool_streams_create(attn_cus, ctypes.byref(sa), ctypes.byref(sf)))
        _pool_streams[key] = (torch.cuda.ExternalStream(sa.value, device=d),
                              torch.cuda.ExternalStream(sf.value, device=d))
    return _pool_streams[key]


def af_pipeline_step(a, w, logits, k: int, mb_sizes, L: int = 1, y=None, stream_a=None,
                     stream_f=None, ws=None, split_tokens: int = 0, join: bool = True):
    """Interleaved A/F layer step(s); returns y [B, Hq*D].

    Without explicit streams the step runs on two side streams that first wait
    for the current stream; with ``join`` the current stream then waits for
    stream_f, so the result is ordered on the caller's stream.
    """
    lib = load()
    if stream_a is None or stream_f is None:
        stream_a, stream_f = pipeline_streams(a.q.device)
        cur = torch.cuda.current_stream(a.q.device)
        stream_a.wait_stream(cur)
        stream_f.wait_stream(cur)
    if y is None:
        y = torch.empty(a.B, a.Hq * a.D, dtype=torch.bfloat16, device=a.q.device)
    aa = attn_args(a, None, split_tokens)
    fa = ffn_args(None, w, y, logits, k)
    M = len(mb_sizes)
    mb = (ctypes.c_int32 * M)(*mb_sizes)
    n = ctypes.c_size_t()
    _check(lib.aflex_af_pipeline_workspace(ctypes.byref(aa), ctypes.byref(fa), M, mb, L,
                                           ctypes.byref(n)))
    p, sz = _ws("pipe", n.value, a.q.device, ws, (stream_a, stream_f))
    _check(lib.aflex_af_pipeline_step(ctypes.byref(aa), ctypes.byref(fa), M, mb, L, p, sz,
                                      _stream(stream_a), _stream(stream_f)))
    if join:
        torch.cuda.current_stream(a.q.device).wait_stream(stream_f)
    return y


def af_layer_step(a, w, layer, k: int, mb_sizes, L: int = 1, y=None, stream_a=None, stream_f=None,
                  ws=None, join: bool = True):
    """The whole decode layer on the interleaved A/F step: per microbatch KV
    append, attention and output projection (+ layer input) on stream_a, the
    MoE block (RMSNorm, router, experts, residual) on stream_f. Appends the
    new K/V into a's pools in place; returns y [B, H]. Streams as for
    af_pipeline_step."""
    lib = load()
    if stream_a is None or stream_f is None:
        stream_a, stream_f = pipeline_streams(a.q.device)
        cur = torch.cuda.current_stream(a.q.device)
        stream_a.wait_stream(cur)
        stream_f.wait_stream(cur)
    if y is None:
        y = torch.empty(a.B, w.H, dtype=torch.bfloat16, device=a.q.device)
    aa = attn_args(a, None)
    fa = ffn_args(None, w, y, None, k)
    la = LayerArgs(k_new=_ptr(layer.k_new), v_new=_ptr(layer.v_new), k_cache=_ptr(a.k_cache),
                   v_cache=_ptr(a.v_cache), w_o=_ptr(layer.w_o), x_in=_ptr(layer.x_in),
                   norm_weight=_ptr(layer.norm_weight), router_weight=_ptr(layer.router_weight),
                   eps=layer.eps)
    M = len(mb_sizes)
    mb = (ctypes.c_int32 * M)(*mb_sizes)
    n = ctypes.c_size_t()
    _check(lib.aflex_af_layer_workspace(ctypes.byref(aa), ctypes.byref(fa), ctypes.byref(la), M, mb, L,
                                        ctypes.byref(n)))
    p, sz = _ws("layer", n.value, a.q.device, ws, (stream_a, stream_f))
    _check(lib.aflex_af_layer_step(ctypes.byref(aa), ctypes.byref(fa), ctypes.byref(la), M, mb, L, p, sz,
                                   _stream(stream_a), _stream(stream_f)))
    if join:
        torch.cuda.current_stream(a.q.device).wait_stream(stream_f)
    return y
