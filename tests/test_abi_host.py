"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function the header declares, and rejects bad arguments with the
documented status before launching anything."""
import ctypes
import os

import pytest

from paper_2608_01891_amd import aflex

FAKE = 0x10000000  # aligned, never dereferenced: validation fails before any launch


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(aflex.LIB_PATH):
        from paper_2608_01891_amd import build
        build.build(verbose=False)
    return aflex.load()


def test_exports_every_declared_symbol(lib):
    names = aflex.exported_names()
    assert len(names) == 25
    for n in names:
        assert hasattr(lib, n), n
    assert lib.aflex_version().startswith(b"aflex")


def test_teardown_with_nothing_cached(lib):
    """The teardown call destroys only what the library created; with nothing
    created yet it succeeds without touching a device, and it may repeat."""
    assert lib.aflex_teardown() == aflex.OK
    assert lib.aflex_teardown() == aflex.OK
    aflex.close()


def _attn(**kw):
    a = aflex.AttnArgs(q=FAKE, k_cache=FAKE, v_cache=FAKE, block_table=FAKE, context_lens=FAKE,
                       out=FAKE, B=4, Hq=8, Hkv=2, D=64, block_size=16, max_blocks_per_seq=13,
                       num_blocks=32, max_context_len=200, scale=0.0, split_tokens=0)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def _ffn(**kw):
    f = aflex.FfnArgs(x=FAKE, router_logits=FAKE, w_gate=FAKE, w_up=FAKE, w_down=FAKE, y=FAKE,
                      T=4, H=512, I=1408, E=8, k=2)
    for k, v in kw.items():
        setattr(f, k, v)
    return f


def _attn_status(lib, a, ws_bytes=1 << 40):
    return lib.aflex_attn_decode(ctypes.byref(a), ctypes.c_void_p(FAKE), ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), aflex.ERR_INVALID_ARG),
    (dict(out=None), aflex.ERR_INVALID_ARG),
    (dict(B=0), aflex.ERR_INVALID_ARG),
    (dict(Hq=6, Hkv=4), aflex.ERR_INVALID_ARG),
    (dict(D=96), aflex.ERR_UNSUPPORTED),
    (dict(block_size=32), aflex.ERR_UNSUPPORTED),
    (dict(Hq=34, Hkv=2), aflex.ERR_UNSUPPORTED),
    (dict(max_context_len=209), aflex.ERR_INVALID_ARG),
    (dict(split_tokens=100), aflex.ERR_INVALID_ARG),
    (dict(split_tokens=2048), aflex.ERR_INVALID_ARG),
    (dict(scale=float("nan")), aflex.ERR_INVALID_ARG),
    (dict(q=FAKE + 2), aflex.ERR_ALIGNMENT),
    (dict(block_table=FAKE + 2), aflex.ERR_ALIGNMENT),
])
def test_attention_rejects(lib, kw, status):
    assert _attn_status(lib, _attn(**kw)) == status
    assert lib.aflex_last_error()


def test_attention_noalloc_rejects_before_launch(lib):
    """The no-allocation attention validates like aflex_attn_decode and refuses
    shapes whose split partials exceed its static scratch (64 MiB), on the host,
    before any device call."""
    a = _attn(q=None)
    assert lib.aflex_attn_decode_noalloc(ctypes.byref(a), None) == aflex.ERR_INVALID_ARG
    big = _attn(B=4096, Hq=64, Hkv=8, D=128, max_blocks_per_seq=2048, max_context_len=32768)
    assert lib.aflex_attn_decode_noalloc(ctypes.byref(big), None) == aflex.ERR_WORKSPACE
    assert b"static scratch" in lib.aflex_last_error()


def test_attention_workspace(lib):
    n = ctypes.c_size_t()
    a = _attn()
    assert lib.aflex_attn_decode_workspace(ctypes.byref(a), ctypes.byref(n)) == aflex.OK
    small = n.value
    a = _attn(max_blocks_per_seq=512, max_context_len=8192, B=64, Hq=64, Hkv=8, D=128)
    assert lib.aflex_attn_decode_workspace(ctypes.byref(a), ctypes.byref(n)) == aflex.OK
    # fp32 partials (O, m, l) of up to one piece per (sequence, kv head) pair
    # plus one per work-group (768 on a 256-CU device), one merge counter per pair
    assert n.value >= (64 * 8 + 768) * 8 * (128 + 2) * 4 + 64 * 8 * 8 > small
    assert _attn_status(lib, a, ws_bytes=n.value - 1) == aflex.ERR_WORKSPACE
    assert b"workspace" in lib.aflex_last_error()
    assert lib.aflex_attn_decode(ctypes.byref(a), ctypes.c_void_p(FAKE + 128), n.value,
                                 None) == aflex.ERR_ALIGNMENT


@pytest.mark.parametrize("kw,moe,status", [
    (dict(H=500), False, aflex.ERR_UNSUPPORTED),
    (dict(I=100), False, aflex.ERR_UNSUPPORTED),
    (dict(T=0), False, aflex.ERR_INVALID_ARG),
    (dict(w_down=None), False, aflex.ERR_INVALID_ARG),
    (dict(y=FAKE + 8), False, aflex.ERR_ALIGNMENT),
    (dict(k=3, E=2), True, aflex.ERR_INVALID_ARG),
    (dict(k=0), True, aflex.ERR_INVALID_ARG),
    (dict(E=65), True, aflex.ERR_UNSUPPORTED),
    (dict(E=16, k=9), True, aflex.ERR_UNSUPPORTED),
    (dict(router_logits=None), True, aflex.ERR_INVALID_ARG),
])
def test_ffn_rejects(lib, kw, moe, status):
    f = _ffn(**kw)
    fn = lib.aflex_moe_ffn if moe else lib.aflex_ffn_swiglu
    assert fn(ctypes.byref(f), ctypes.c_void_p(FAKE), 1 << 40, None) == status


def test_ffn_workspaces(lib):
    n = ctypes.c_size_t()
    f = _ffn(T=512, H=5120, I=25600)
    assert lib.aflex_ffn_swiglu_workspace(ctypes.byref(f), ctypes.byref(n)) == aflex.OK
    assert n.value >= 512 * 25600 * 2
    f = _ffn(T=256, H=4096, I=14336)
    assert lib.aflex_moe_ffn_workspace(ctypes.byref(f), ctypes.byref(n)) == aflex.OK
    assert n.value >= 512 * 14336 * 2 + 512 * 4096 * 4
    assert lib.aflex_moe_ffn(ctypes.byref(f), ctypes.c_void_p(FAKE), n.value - 256,
                             None) == aflex.ERR_WORKSPACE


def test_pipeline_rejects(lib):
    a = _attn(B=8, Hq=4, Hkv=2, D=64)
    f = _ffn(x=None, T=8, H=256, I=128, E=4, k=2)
    mb = (ctypes.c_int32 * 2)(3, 5)
    n = ctypes.c_size_t()
    assert lib.aflex_af_pipeline_workspace(ctypes.byref(a), ctypes.byref(f), 2, mb, 1,
                                           ctypes.byref(n)) == aflex.OK
    step = lambda a, f, M, mb, L, sa=FAKE, sf=FAKE + 64: lib.aflex_af_pipeline_step(
        ctypes.byref(a), ctypes.byref(f), M, mb, L, ctypes.c_void_p(FAKE), 1 << 40,
        ctypes.c_void_p(sa), ctypes.c_void_p(sf))
    assert step(a, f, 2, (ctypes.c_int32 * 2)(3, 4), 1) == aflex.ERR_INVALID_ARG  # sum != B
    assert step(a, f, 0, mb, 1) == aflex.ERR_INVALID_ARG
    assert step(a, f, 2, mb, 0) == aflex.ERR_INVALID_ARG
    assert step(a, f, 2, (ctypes.c_int32 * 2)(0, 8), 1) == aflex.ERR_INVALID_ARG
    assert step(a, _ffn(x=None, T=8, H=512, I=128, E=4, k=2), 2, mb, 1) == aflex.ERR_INVALID_ARG
    assert step(a, f, 2, mb, 1, sa=FAKE, sf=FAKE) == aflex.ERR_INVALID_ARG
    assert b"differ" in lib.aflex_last_error()
    assert lib.aflex_af_pipeline_step(ctypes.byref(a), ctypes.byref(f), 2, mb, 1,
                                      ctypes.c_void_p(FAKE), n.value - 1, None,
                                      ctypes.c_void_p(FAKE)) == aflex.ERR_WORKSPACE


def _prefill(**kw):
    a = aflex.PrefillArgs(q=FAKE, k=FAKE, v=FAKE, cu_seqlens=FAKE, out=FAKE, B=2, T=100, Hq=8, Hkv=2,
                          D=128, max_seqlen=60, scale=0.0)
    for k, v in kw.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), aflex.ERR_INVALID_ARG),
    (dict(cu_seqlens=None), aflex.ERR_INVALID_ARG),
    (dict(B=0), aflex.ERR_INVALID_ARG),
    (dict(T=-1), aflex.ERR_INVALID_ARG),
    (dict(Hq=6, Hkv=4), aflex.ERR_INVALID_ARG),
    (dict(D=64), aflex.ERR_UNSUPPORTED),
    (dict(B=70000), aflex.ERR_UNSUPPORTED),
    (dict(max_seqlen=101), aflex.ERR_INVALID_ARG),
    (dict(max_seqlen=-1), aflex.ERR_INVALID_ARG),
    (dict(scale=float("nan")), aflex.ERR_INVALID_ARG),
    (dict(out=FAKE + 8), aflex.ERR_ALIGNMENT),
    (dict(cu_seqlens=FAKE + 2), aflex.ERR_ALIGNMENT),
])
def test_prefill_validation(lib, kw, status):
    a = _prefill(**kw)
    assert lib.aflex_attn_prefill(ctypes.byref(a), None) == status
    assert lib.aflex_last_error().startswith(b"prefill")


def test_kv_write_validation(lib):
    def mk(**kw):
        a = aflex.KvWriteArgs(k_new=FAKE, v_new=FAKE, cu_seqlens=FAKE, k_cache=FAKE, v_cache=FAKE,
                              block_table=FAKE, context_lens=FAKE, B=2, T=40, Hkv=2, D=128, max_seqlen=30,
                              block_size=16, max_blocks_per_seq=4, num_blocks=8)
        for k, v in kw.items():
            setattr(a, k, v)
        return a
    for kw, st in [(dict(k_new=None), aflex.ERR_INVALID_ARG), (dict(max_seqlen=41), aflex.ERR_INVALID_ARG),
                   (dict(D=96), aflex.ERR_UNSUPPORTED), (dict(block_size=8), aflex.ERR_UNSUPPORTED),
                   (dict(Hkv=65), aflex.ERR_UNSUPPORTED), (dict(v_cache=FAKE + 4), aflex.ERR_ALIGNMENT),
                   (dict(cu_seqlens=FAKE + 1), aflex.ERR_ALIGNMENT)]:
        a = mk(**kw)
        assert lib.aflex_kv_write(ctypes.byref(a), None) == st, kw
        assert lib.aflex_last_error().startswith(b"kv_write")


def test_pool_streams_validation(lib):
    sa = ctypes.c_void_p()
    assert lib.aflex_pool_streams_create(128, None, ctypes.byref(sa)) == aflex.ERR_INVALID_ARG
    assert lib.aflex_last_error().startswith(b"pool streams")
    sf = ctypes.c_void_p()
    assert lib.aflex_pool_streams_create(100, ctypes.byref(sa), ctypes.byref(sf)) == aflex.ERR_UNSUPPORTED
    assert sa.value is None and sf.value is None


def _layer_status(lib, a, f, la, M=2, mbs=(2, 2), L=1):
    mb = (ctypes.c_int32 * M)(*mbs)
    n = ctypes.c_size_t()
    return lib.aflex_af_layer_workspace(ctypes.byref(a), ctypes.byref(f), ctypes.byref(la), M, mb, L,
                                        ctypes.byref(n))


@pytest.mark.parametrize("case,status", [
    ("ok", aflex.OK),
    ("dense", aflex.ERR_UNSUPPORTED),
    ("other_pool", aflex.ERR_INVALID_ARG),
    ("no_router", aflex.ERR_INVALID_ARG),
    ("misaligned_wo", aflex.ERR_ALIGNMENT),
    ("L2_hidden_mismatch", aflex.ERR_INVALID_ARG),
    ("bad_eps", aflex.ERR_INVALID_ARG),
])
def test_layer_step_validation(lib, case, status):
    """The decode-layer step validates on the host: the MoE block only (E >= 1),
    the append must target the pools the attention reads, L > 1 needs H = Hq*D."""
    a = _attn(out=None)                       # B=4, Hq=8, Hkv=2, D=64: Hq*D = 512
    f = _ffn(x=None, router_logits=None, H=512, I=1408, E=8, k=2)
    la = aflex.LayerArgs(k_new=FAKE, v_new=FAKE, k_cache=FAKE, v_cache=FAKE, w_o=FAKE, x_in=None,
                         norm_weight=FAKE, router_weight=FAKE, eps=1e-5)
    L = 1
    if case == "dense":
        f.E, f.k = 0, 0
    elif case == "other_pool":
        la.k_cache = FAKE + 256
    elif case == "no_router":
        la.router_weight = None
    elif case == "misaligned_wo":
        la.w_o = FAKE + 2
    elif case == "L2_hidden_mismatch":
        f.H, L = 1024, 2
    elif case == "bad_eps":
        la.eps = -1.0
    assert _layer_status(lib, a, f, la, L=L) == status
