// C-ABI layer of libaflex: host-side validation, workspace queries, launches
// and the two-stream interleaved A/F layer-step driver.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <vector>

#include "aflex.h"
#include "kernels.h"
#include "profile.h"

namespace {

thread_local char g_err[512] = "";

aflex_status fail(aflex_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, status, ...) \
  do {                             \
    if (!(cond)) return fail(status, __VA_ARGS__); \
  } while (0)

aflex_status check_attn(const aflex_attn_args* a, bool need_out) {
  REQUIRE(a, AFLEX_ERR_INVALID_ARG, "attn: args is NULL");
  REQUIRE(a->q && a->k_cache && a->v_cache && a->block_table && a->context_lens, AFLEX_ERR_INVALID_ARG,
          "attn: NULL tensor pointer");
  REQUIRE(!need_out || a->out, AFLEX_ERR_INVALID_ARG, "attn: out is NULL");
  REQUIRE(a->B >= 1 && a->Hq >= 1 && a->Hkv >= 1 && a->D >= 1, AFLEX_ERR_INVALID_ARG,
          "attn: B, Hq, Hkv, D must be positive (got %d, %d, %d, %d)", a->B, a->Hq, a->Hkv, a->D);
  REQUIRE(a->num_blocks >= 1 && a->max_blocks_per_seq >= 1, AFLEX_ERR_INVALID_ARG,
          "attn: num_blocks and max_blocks_per_seq must be positive");
  REQUIRE(a->max_context_len >= 0, AFLEX_ERR_INVALID_ARG, "attn: max_context_len < 0");
  REQUIRE(a->Hq % a->Hkv == 0, AFLEX_ERR_INVALID_ARG, "attn: Hq (%d) not a multiple of Hkv (%d)", a->Hq, a->Hkv);
  REQUIRE(a->D == 64 || a->D == 128, AFLEX_ERR_UNSUPPORTED, "attn: head_dim %d unsupported (64 or 128)", a->D);
  REQUIRE(a->block_size == 16, AFLEX_ERR_UNSUPPORTED, "attn: block_size %d unsupported (16)", a->block_size);
  REQUIRE(a->Hq / a->Hkv <= 16, AFLEX_ERR_UNSUPPORTED, "attn: %d query heads per kv head (max 16)",
          a->Hq / a->Hkv);
  REQUIRE((long long)a->max_context_len <= (long long)a->max_blocks_per_seq * a->block_size,
          AFLEX_ERR_INVALID_ARG, "attn: max_context_len %d exceeds the block table capacity %lld",
          a->max_context_len, (long long)a->max_blocks_per_seq * a->block_size);
  REQUIRE(a->split_tokens == 0 || (a->split_tokens % 128 == 0 && a->split_tokens >= 128 &&
                                   a->split_tokens <= 1024),
          AFLEX_ERR_INVALID_ARG, "attn: split_tokens %d must be 0 or a multiple of 128 in [128, 1024]",
          a->split_tokens);
  REQUIRE(isfinite(a->scale) && a->scale >= 0.f, AFLEX_ERR_INVALID_ARG, "attn: scale must be finite and >= 0");
  REQUIRE(aflex::attn_shape_fits(*a), AFLEX_ERR_UNSUPPORTED,
          "attn: B * Hkv * ceil(max_context_len / 16) must stay below 2^30");
  REQUIRE(aligned16(a->q) && aligned16(a->k_cache) && aligned16(a->v_cache) && (!a->out || aligned16(a->out)),
          AFLEX_ERR_ALIGNMENT, "attn: q, k_cache, v_cache and out must be 16-byte aligned");
  REQUIRE(((uintptr_t)a->block_table & 3u) == 0 && ((uintptr_t)a->context_lens & 3u) == 0, AFLEX_ERR_ALIGNMENT,
          "attn: block_table and context_lens must be 4-byte aligned");
  return AFLEX_OK;
}

aflex_status check_ffn(const aflex_ffn_args* f, bool moe, bool need_x) {
  const char* who = moe ? "moe" : "swiglu";
  REQUIRE(f, AFLEX_ERR_INVALID_ARG, "%s: args is NULL", who);
  REQUIRE((!need_x || f->x) && f->w_gate && f->w_up && f->w_down && f->y, AFLEX_ERR_INVALID_ARG,
          "%s: NULL tensor pointer", who);
  REQUIRE(f->T >= 1 && f->H >= 1 && f->I >= 1, AFLEX_ERR_INVALID_ARG, "%s: T, H, I must be positive", who);
  REQUIRE(f->H % 64 == 0 && f->I % 64 == 0, AFLEX_ERR_UNSUPPORTED, "%s: H (%d) and I (%d) must be multiples of 64",
          who, f->H, f->I);
  REQUIRE((!f->x || aligned16(f->x)) && aligned16(f->w_gate) && aligned16(f->w_up) && aligned16(f->w_down) &&
              aligned16(f->y),
          AFLEX_ERR_ALIGNMENT, "%s: tensors must be 16-byte aligned", who);
  if (moe) {
    REQUIRE(f->router_logits, AFLEX_ERR_INVALID_ARG, "moe: router_logits is NULL");
    REQUIRE(f->E >= 1 && f->k >= 1 && f->k <= f->E, AFLEX_ERR_INVALID_ARG, "moe: need 1 <= k <= E (k=%d, E=%d)",
            f->k, f->E);
    REQUIRE(f->E <= 64 && f->k <= 8, AFLEX_ERR_UNSUPPORTED, "moe: E <= 64 and k <= 8 supported (E=%d, k=%d)", f->E,
            f->k);
    REQUIRE((long long)f->T * f->k < (1ll << 30), AFLEX_ERR_UNSUPPORTED, "moe: too many token/slot pairs");
  }
  return AFLEX_OK;
}

aflex_status check_ws(void* ws, size_t have, size_t need, const char* who) {
  REQUIRE(have >= need, AFLEX_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu required", who, have, need);
  REQUIRE(need == 0 || ws, AFLEX_ERR_WORKSPACE, "%s: workspace is NULL", who);
  REQUIRE(((uintptr_t)ws & 255u) == 0, AFLEX_ERR_ALIGNMENT, "%s: workspace must be 256-byte aligned", who);
  return AFLEX_OK;
}

aflex_status hip_status(hipError_t e, const char* who) {
  if (e == hipSuccess) return AFLEX_OK;
  return fail(AFLEX_ERR_HIP, "%s: HIP error %d (%s)", who, (int)e, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Pipeline driver.
struct PipeLayout {
  size_t attn_out, attn_ws, route_ws, route_stride, ffn_ws, total;
};

aflex_attn_args mb_attn(const aflex_attn_args& a, int off, int n) {
  aflex_attn_args m = a;
  m.B = n;
  m.q = a.q + (size_t)off * a.Hq * a.D;
  m.block_table = a.block_table + (size_t)off * a.max_blocks_per_seq;
  m.context_lens = a.context_lens + off;
  m.out = a.out ? a.out + (size_t)off * a.Hq * a.D : nullptr;
  return m;
}

aflex_ffn_args mb_ffn(const aflex_ffn_args& f, int off, int n) {
  aflex_ffn_args m = f;
  m.T = n;
  m.x = f.x ? f.x + (size_t)off * f.H : nullptr;
  m.y = f.y + (size_t)off * f.H;
  m.router_logits = f.router_logits ? f.router_logits + (size_t)off * f.E : nullptr;
  m.topk_ids = nullptr;
  m.topk_w = nullptr;
  m.expert_offsets = nullptr;
  m.sorted_pairs = nullptr;
  return m;
}

PipeLayout pipe_layout(const aflex_attn_args& a, const aflex_ffn_args& f, int M, const int32_t* mb) {
  PipeLayout L;
  size_t aw = 0, fw = 0, rw = 0;
  int off = 0;
  for (int i = 0; i < M; ++i) {
    aflex_attn_args am = mb_attn(a, off, mb[i]);
    aflex_ffn_args fm = mb_ffn(f, off, mb[i]);
    size_t x = aflex::attn_workspace_bytes(am);
    size_t y = f.E ? aflex::moe_expert_bytes(fm) : aflex::swiglu_workspace_bytes(fm);
    size_t z = f.E ? aflex::moe_route_bytes(fm) : 0;
    aw = x > aw ? x : aw;
    fw = y > fw ? y : fw;
    rw = z > rw ? z : rw;
    off += mb[i];
  }
  L.attn_out = 0;
  L.attn_ws = aflex::align_up((size_t)a.B * a.Hq * a.D * 2, 256);
  L.route_ws = L.attn_ws + aflex::align_up(aw, 256);
  L.route_stride = aflex::align_up(rw, 256);
  L.ffn_ws = L.route_ws + (size_t)M * L.route_stride;
  L.total = L.ffn_ws + aflex::align_up(fw, 256);
  return L;
}

aflex_status check_pipe(const aflex_attn_args* a, const aflex_ffn_args* f, int32_t M, const int32_t* mb, int32_t L) {
  aflex_status s = check_attn(a, false);
  if (s != AFLEX_OK) return s;
  s = check_ffn(f, f && f->E > 0, false);
  if (s != AFLEX_OK) return s;
  REQUIRE(M >= 1 && M <= 64, AFLEX_ERR_INVALID_ARG, "pipeline: M=%d must be in [1, 64]", M);
  REQUIRE(mb, AFLEX_ERR_INVALID_ARG, "pipeline: mb_sizes is NULL");
  REQUIRE(L >= 1, AFLEX_ERR_INVALID_ARG, "pipeline: L=%d must be >= 1", L);
  long long sum = 0;
  for (int i = 0; i < M; ++i) {
    REQUIRE(mb[i] >= 1, AFLEX_ERR_INVALID_ARG, "pipeline: mb_sizes[%d]=%d must be >= 1", i, mb[i]);
    sum += mb[i];
  }
  REQUIRE(sum == a->B, AFLEX_ERR_INVALID_ARG, "pipeline: sum of mb_sizes %lld != B %d", sum, a->B);
  REQUIRE(f->T == a->B, AFLEX_ERR_INVALID_ARG, "pipeline: ffn T %d != attention B %d", f->T, a->B);
  REQUIRE(f->H == a->Hq * a->D, AFLEX_ERR_INVALID_ARG, "pipeline: ffn H %d != Hq*D %d", f->H, a->Hq * a->D);
  return AFLEX_OK;
}

struct EventPool {
  std::mutex mu;
  std::vector<std::vector<hipEvent_t>> per_device;
};
EventPool g_events;

// At least `need` events of the current device for ordering the two streams
// of a step (created on first use, kept for later calls). The caller holds
// g_events.mu for as long as it records and waits on them.
aflex_status pipeline_events(size_t need, std::vector<hipEvent_t>** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "pipeline");
  if ((int)g_events.per_device.size() <= dev) g_events.per_device.resize(dev + 1);
  std::vector<hipEvent_t>& ev = g_events.per_device[dev];
  while (ev.size() < need) {
    hipEvent_t x;
    e = hipEventCreateWithFlags(&x, hipEventDisableTiming);
    if (e != hipSuccess) return hip_status(e, "pipeline: event create");
    ev.push_back(x);
  }
  *out = &ev;
  return AFLEX_OK;
}

// ---------------------------------------------------------------------------
// Whole decode layer on the two streams.
struct LayerLayout {
  size_t attn_out, h, attn_ws, lin_ws, blk_ws, total;
};

aflex_linear_args mb_linear(const aflex_attn_args& a, const aflex_ffn_args& f, const aflex_layer_args& ly,
                            const uint16_t* x, uint16_t* y, int n) {
  aflex_linear_args l;
  l.x = x;
  l.w = ly.w_o;
  l.y = y;
  l.T = n;
  l.K = a.Hq * a.D;
  l.N = f.H;
  return l;
}

aflex_moe_block_args mb_block(const aflex_ffn_args& f, const aflex_layer_args& ly, int off, int n,
                              const uint16_t* h) {
  aflex_moe_block_args m;
  m.ffn = mb_ffn(f, off, n);
  m.ffn.x = h;
  m.ffn.router_logits = nullptr;
  m.norm_weight = ly.norm_weight;
  m.router_weight = ly.router_weight;
  m.eps = ly.eps;
  m.residual = 1;
  m.router_logits_out = nullptr;
  return m;
}

LayerLayout layer_layout(const aflex_attn_args& a, const aflex_ffn_args& f, const aflex_layer_args& ly, int M,
                         const int32_t* mb) {
  LayerLayout L;
  size_t aw = 0, lw = 0, bw = 0;
  int off = 0;
  for (int i = 0; i < M; ++i) {
    const size_t x = aflex::attn_workspace_bytes(mb_attn(a, off, mb[i]));
    const size_t y = aflex::linear_workspace_bytes(mb_linear(a, f, ly, nullptr, nullptr, mb[i]));
    const size_t z = aflex::moe_block_workspace_bytes(mb_block(f, ly, off, mb[i], nullptr));
    aw = x > aw ? x : aw;
    lw = y > lw ? y : lw;
    bw = z > bw ? z : bw;
    off += mb[i];
  }
  L.attn_out = 0;
  L.h = aflex::align_up((size_t)a.B * a.Hq * a.D * 2, 256);
  L.attn_ws = L.h + aflex::align_up((size_t)a.B * f.H * 2, 256);
  L.lin_ws = L.attn_ws + aflex::align_up(aw, 256);
  L.blk_ws = L.lin_ws + aflex::align_up(lw, 256);
  L.total = L.blk_ws + aflex::align_up(bw, 256);
  return L;
}

aflex_status check_layer(const aflex_attn_args* a, const aflex_ffn_args* f, const aflex_layer_args* ly, int32_t M,
                         const int32_t* mb, int32_t L) {
  aflex_status s = check_attn(a, false);
  if (s != AFLEX_OK) return s;
  REQUIRE(f, AFLEX_ERR_INVALID_ARG, "layer: ffn args is NULL");
  REQUIRE(ly, AFLEX_ERR_INVALID_ARG, "layer: layer args is NULL");
  REQUIRE(f->E >= 1, AFLEX_ERR_UNSUPPORTED, "layer: the decode layer step runs the MoE block (E >= 1)");
  aflex_ffn_args fc = *f;
  fc.router_logits = reinterpret_cast<const float*>(ly->router_weight);  // computed: only non-NULL matters
  s = check_ffn(&fc, true, false);
  if (s != AFLEX_OK) return s;
  REQUIRE(ly->k_new && ly->v_new && ly->k_cache && ly->v_cache && ly->w_o && ly->norm_weight && ly->router_weight,
          AFLEX_ERR_INVALID_ARG, "layer: NULL tensor pointer");
  REQUIRE(ly->k_cache == a->k_cache && ly->v_cache == a->v_cache, AFLEX_ERR_INVALID_ARG,
          "layer: k_cache / v_cache must be the pools the attention reads");
  REQUIRE(isfinite(ly->eps) && ly->eps >= 0.f, AFLEX_ERR_INVALID_ARG, "layer: eps must be finite and >= 0");
  REQUIRE(f->H <= 16384, AFLEX_ERR_UNSUPPORTED, "layer: H=%d above 16384", f->H);
  REQUIRE(aligned16(ly->k_new) && aligned16(ly->v_new) && aligned16(ly->w_o) && aligned16(ly->norm_weight) &&
              aligned16(ly->router_weight) && (!ly->x_in || aligned16(ly->x_in)),
          AFLEX_ERR_ALIGNMENT, "layer: tensors must be 16-byte aligned");
  REQUIRE(M >= 1 && M <= 64, AFLEX_ERR_INVALID_ARG, "layer: M=%d must be in [1, 64]", M);
  REQUIRE(mb, AFLEX_ERR_INVALID_ARG, "layer: mb_sizes is NULL");
  REQUIRE(L >= 1, AFLEX_ERR_INVALID_ARG, "layer: L=%d must be >= 1", L);
  long long sum = 0;
  for (int i = 0; i < M; ++i) {
    REQUIRE(mb[i] >= 1, AFLEX_ERR_INVALID_ARG, "layer: mb_sizes[%d]=%d must be >= 1", i, mb[i]);
    sum += mb[i];
  }
  REQUIRE(sum == a->B, AFLEX_ERR_INVALID_ARG, "layer: sum of mb_sizes %lld != B %d", sum, a->B);
  REQUIRE(f->T == a->B, AFLEX_ERR_INVALID_ARG, "layer: ffn T %d != attention B %d", f->T, a->B);
  REQUIRE(L == 1 || f->H == a->Hq * a->D, AFLEX_ERR_INVALID_ARG,
          "layer: L > 1 feeds y back as q, so H (%d) must equal Hq*D (%d)", f->H, a->Hq * a->D);
  return AFLEX_OK;
}

}  // namespace

extern "C" {

const char* aflex_last_error(void) { return g_err; }

aflex_status aflex_kv_append(const aflex_kv_append_args* a, aflex_stream stream) {
  REQUIRE(a, AFLEX_ERR_INVALID_ARG, "kv_append: args is NULL");
  REQUIRE(a->k_new && a->v_new && a->k_cache && a->v_cache && a->block_table && a->context_lens,
          AFLEX_ERR_INVALID_ARG, "kv_append: NULL tensor pointer");
  REQUIRE(a->B >= 1 && a->Hkv >= 1 && a->num_blocks >= 1 && a->max_blocks_per_seq >= 1, AFLEX_ERR_INVALID_ARG,
          "kv_append: B, Hkv, num_blocks, max_blocks_per_seq must be positive");
  REQUIRE(a->D == 64 || a->D == 128, AFLEX_ERR_UNSUPPORTED, "kv_append: head_dim %d unsupported (64 or 128)", a->D);
  REQUIRE(a->block_size == 16, AFLEX_ERR_UNSUPPORTED, "kv_append: block_size %d unsupported (16)", a->block_size);
  REQUIRE(aligned16(a->k_new) && aligned16(a->v_new) && aligned16(a->k_cache) && aligned16(a->v_cache),
          AFLEX_ERR_ALIGNMENT, "kv_append: tensors must be 16-byte aligned");
  return hip_status(aflex::launch_kv_append(*a, (hipStream_t)stream), "kv_append");
}

aflex_status aflex_pool_streams_create(int32_t attn_cus, aflex_stream* stream_a, aflex_stream* stream_f) {
  REQUIRE(stream_a && stream_f, AFLEX_ERR_INVALID_ARG, "pool streams: NULL output");
  *stream_a = nullptr;
  *stream_f = nullptr;
  REQUIRE(attn_cus == 64 || attn_cus == 128 || attn_cus == 192, AFLEX_ERR_UNSUPPORTED,
          "pool streams: attn_cus %d must be 64, 128 or 192", attn_cus);
  int dev = 0, ncu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e, "pool streams");
  REQUIRE(ncu == 256, AFLEX_ERR_UNSUPPORTED, "pool streams: device has %d CUs (256 expected)", ncu);
  uint32_t ma[8] = {0}, mf[8] = {0};
  for (int i = 0; i < 256; ++i) {
    if ((i / 8) % 4 < attn_cus / 64)
      ma[i / 32] |= 1u << (i % 32);
    else
      mf[i / 32] |= 1u << (i % 32);
  }
  hipStream_t sa = nullptr, sf = nullptr;
  e = hipExtStreamCreateWithCUMask(&sa, 8, ma);
  if (e == hipSuccess) e = hipExtStreamCreateWithCUMask(&sf, 8, mf);
  if (e != hipSuccess) {
    if (sa) (void)hipStreamDestroy(sa);
    return hip_status(e, "pool streams");
  }
  *stream_a = sa;
  *stream_f = sf;
  return AFLEX_OK;
}

aflex_status aflex_pool_streams_destroy(aflex_stream stream_a, aflex_stream stream_f) {
  hipError_t e = hipSuccess;
  if (stream_a) e = hipStreamDestroy((hipStream_t)stream_a);
  if (stream_f) {
    const hipError_t e2 = hipStreamDestroy((hipStream_t)stream_f);
    if (e == hipSuccess) e = e2;
  }
  return hip_status(e, "pool streams");
}

aflex_status aflex_kv_write(const aflex_kv_write_args* a, aflex_stream stream) {
  REQUIRE(a, AFLEX_ERR_INVALID_ARG, "kv_write: args is NULL");
  REQUIRE(a->k_new && a->v_new && a->cu_seqlens && a->k_cache && a->v_cache && a->block_table && a->context_lens,
          AFLEX_ERR_INVALID_ARG, "kv_write: NULL tensor pointer");
  REQUIRE(a->B >= 1 && a->T >= 0 && a->Hkv >= 1 && a->num_blocks >= 1 && a->max_blocks_per_seq >= 1 &&
              a->max_seqlen >= 0,
          AFLEX_ERR_INVALID_ARG, "kv_write: need B, Hkv, num_blocks, max_blocks_per_seq >= 1 and T, max_seqlen >= 0");
  REQUIRE(a->max_seqlen <= a->T, AFLEX_ERR_INVALID_ARG, "kv_write: max_seqlen %d exceeds T %d", a->max_seqlen, a->T);
  REQUIRE(a->D == 64 || a->D == 128, AFLEX_ERR_UNSUPPORTED, "kv_write: head_dim %d unsupported (64 or 128)", a->D);
  REQUIRE(a->block_size == 16, AFLEX_ERR_UNSUPPORTED, "kv_write: block_size %d unsupported (16)", a->block_size);
  REQUIRE(a->Hkv * (a->D / 8) <= 1024 && a->B <= 65535, AFLEX_ERR_UNSUPPORTED,
          "kv_write: Hkv * D / 8 must be <= 1024 and B <= 65535");
  REQUIRE(aligned16(a->k_new) && aligned16(a->v_new) && aligned16(a->k_cache) && aligned16(a->v_cache),
          AFLEX_ERR_ALIGNMENT, "kv_write: tensors must be 16-byte aligned");
  REQUIRE(((uintptr_t)a->cu_seqlens & 3u) == 0 && ((uintptr_t)a->block_table & 3u) == 0 &&
              ((uintptr_t)a->context_lens & 3u) == 0,
          AFLEX_ERR_ALIGNMENT, "kv_write: index arrays must be 4-byte aligned");
  return hip_status(aflex::launch_kv_write(*a, (hipStream_t)stream), "kv_write");
}

aflex_status aflex_attn_prefill(const aflex_prefill_args* a, aflex_stream stream) {
  REQUIRE(a, AFLEX_ERR_INVALID_ARG, "prefill: args is NULL");
  REQUIRE(a->q && a->k && a->v && a->cu_seqlens && a->out, AFLEX_ERR_INVALID_ARG, "prefill: NULL tensor pointer");
  REQUIRE(a->B >= 1 && a->T >= 0 && a->Hq >= 1 && a->Hkv >= 1 && a->max_seqlen >= 0, AFLEX_ERR_INVALID_ARG,
          "prefill: need B, Hq, Hkv >= 1 and T, max_seqlen >= 0");
  REQUIRE(a->Hq % a->Hkv == 0, AFLEX_ERR_INVALID_ARG, "prefill: Hq (%d) not a multiple of Hkv (%d)", a->Hq, a->Hkv);
  REQUIRE(a->D == 128, AFLEX_ERR_UNSUPPORTED, "prefill: head_dim %d unsupported (128)", a->D);
  REQUIRE(a->B <= 65535, AFLEX_ERR_UNSUPPORTED, "prefill: B %d above 65535", a->B);
  REQUIRE(a->max_seqlen <= a->T, AFLEX_ERR_INVALID_ARG, "prefill: max_seqlen %d exceeds T %d", a->max_seqlen,
          a->T);
  REQUIRE(isfinite(a->scale) && a->scale >= 0.f, AFLEX_ERR_INVALID_ARG, "prefill: scale must be finite and >= 0");
  REQUIRE(aligned16(a->q) && aligned16(a->k) && aligned16(a->v) && aligned16(a->out), AFLEX_ERR_ALIGNMENT,
          "prefill: q, k, v and out must be 16-byte aligned");
  REQUIRE(((uintptr_t)a->cu_seqlens & 3u) == 0, AFLEX_ERR_ALIGNMENT, "prefill: cu_seqlens must be 4-byte aligned");
  return hip_status(aflex::launch_attn_prefill(*a, (hipStream_t)stream), "prefill");
}

static aflex_status check_linear(const aflex_linear_args* l) {
  REQUIRE(l, AFLEX_ERR_INVALID_ARG, "linear: args is NULL");
  REQUIRE(l->x && l->w && l->y, AFLEX_ERR_INVALID_ARG, "linear: NULL tensor pointer");
  REQUIRE(l->T >= 1 && l->K >= 1 && l->N >= 1, AFLEX_ERR_INVALID_ARG, "linear: T, K, N must be positive");
  REQUIRE(l->K % 64 == 0 && l->N % 64 == 0, AFLEX_ERR_UNSUPPORTED, "linear: K (%d) and N (%d) must be multiples of 64",
          l->K, l->N);
  REQUIRE(aligned16(l->x) && aligned16(l->w) && aligned16(l->y), AFLEX_ERR_ALIGNMENT,
          "linear: tensors must be 16-byte aligned");
  return AFLEX_OK;
}

aflex_status aflex_linear_workspace(const aflex_linear_args* l, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "linear: bytes is NULL");
  aflex_status s = check_linear(l);
  if (s != AFLEX_OK) return s;
  *bytes = aflex::linear_workspace_bytes(*l);
  return AFLEX_OK;
}

aflex_status aflex_linear(const aflex_linear_args* l, void* ws, size_t ws_bytes, aflex_stream stream) {
  aflex_status s = check_linear(l);
  if (s != AFLEX_OK) return s;
  s = check_ws(ws, ws_bytes, aflex::linear_workspace_bytes(*l), "linear");
  if (s != AFLEX_OK) return s;
  return hip_status(aflex::launch_linear(*l, ws, (hipStream_t)stream), "linear");
}
const char* aflex_version(void) { return "aflex 0.2 gfx950"; }

aflex_status aflex_teardown(void) {
  hipError_t first = hipSuccess;
  {
    std::lock_guard<std::mutex> lock(g_events.mu);
    int cur = 0;
    const bool have_cur = hipGetDevice(&cur) == hipSuccess;
    for (size_t dev = 0; dev < g_events.per_device.size(); ++dev) {
      std::vector<hipEvent_t>& ev = g_events.per_device[dev];
      if (ev.empty()) continue;
      hipError_t e = hipSetDevice((int)dev);
      for (hipEvent_t x : ev) {
        const hipError_t r = hipEventDestroy(x);
        if (e == hipSuccess) e = r;
      }
      ev.clear();
      if (first == hipSuccess) first = e;
    }
    if (have_cur) (void)hipSetDevice(cur);
  }
  const hipError_t e = aflex::profile_release();
  if (first == hipSuccess) first = e;
  return hip_status(first, "teardown");
}

aflex_status aflex_attn_decode_workspace(const aflex_attn_args* a, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "attn: bytes is NULL");
  aflex_status s = check_attn(a, false);
  if (s != AFLEX_OK) return s;
  *bytes = aflex::attn_workspace_bytes(*a);
  return AFLEX_OK;
}

aflex_status aflex_attn_decode(const aflex_attn_args* a, void* ws, size_t ws_bytes, aflex_stream stream) {
  aflex_status s = check_attn(a, true);
  if (s != AFLEX_OK) return s;
  s = check_ws(ws, ws_bytes, aflex::attn_workspace_bytes(*a), "attn");
  if (s != AFLEX_OK) return s;
  return hip_status(aflex::launch_attn_decode(*a, ws, (hipStream_t)stream), "attn");
}

aflex_status aflex_attn_decode_noalloc(const aflex_attn_args* a, aflex_stream stream) {
  aflex_status s = check_attn(a, true);
  if (s != AFLEX_OK) return s;
  const size_t need = aflex::attn_workspace_bytes(*a);
  REQUIRE(need <= aflex::kStaticScratchBytes, AFLEX_ERR_WORKSPACE,
          "attn_noalloc: this shape needs %zu bytes of scratch, the library's static scratch holds %zu "
          "(lower B * Hq * ceil(max_context_len / split) or use aflex_attn_decode with a workspace)",
          need, aflex::kStaticScratchBytes);
  void* ws = nullptr;
  hipError_t e = aflex::static_scratch(&ws);
  if (e != hipSuccess) return hip_status(e, "attn_noalloc: static scratch");
  return hip_status(aflex::launch_attn_decode(*a, ws, (hipStream_t)stream), "attn_noalloc");
}

aflex_status aflex_ffn_swiglu_workspace(const aflex_ffn_args* f, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "swiglu: bytes is NULL");
  aflex_status s = check_ffn(f, false, true);
  if (s != AFLEX_OK) return s;
  *bytes = aflex::swiglu_workspace_bytes(*f);
  return AFLEX_OK;
}

aflex_status aflex_ffn_swiglu(const aflex_ffn_args* f, void* ws, size_t ws_bytes, aflex_stream stream) {
  aflex_status s = check_ffn(f, false, true);
  if (s != AFLEX_OK) return s;
  s = check_ws(ws, ws_bytes, aflex::swiglu_workspace_bytes(*f), "swiglu");
  if (s != AFLEX_OK) return s;
  return hip_status(aflex::launch_swiglu(*f, ws, (hipStream_t)stream), "swiglu");
}

aflex_status aflex_moe_ffn_workspace(const aflex_ffn_args* f, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "moe: bytes is NULL");
  aflex_status s = check_ffn(f, true, true);
  if (s != AFLEX_OK) return s;
  *bytes = aflex::moe_workspace_bytes(*f);
  return AFLEX_OK;
}

aflex_status aflex_moe_ffn(const aflex_ffn_args* f, void* ws, size_t ws_bytes, aflex_stream stream) {
  aflex_status s = check_ffn(f, true, true);
  if (s != AFLEX_OK) return s;
  s = check_ws(ws, ws_bytes, aflex::moe_workspace_bytes(*f), "moe");
  if (s != AFLEX_OK) return s;
  return hip_status(aflex::launch_moe(*f, ws, (hipStream_t)stream), "moe");
}

static aflex_status check_moe_block(const aflex_moe_block_args* m) {
  REQUIRE(m, AFLEX_ERR_INVALID_ARG, "moe_block: args is NULL");
  REQUIRE(m->norm_weight && m->router_weight, AFLEX_ERR_INVALID_ARG, "moe_block: NULL norm or router weight");
  REQUIRE(isfinite(m->eps) && m->eps >= 0.f, AFLEX_ERR_INVALID_ARG, "moe_block: eps must be finite and >= 0");
  aflex_ffn_args f = m->ffn;
  f.router_logits = reinterpret_cast<const float*>(m->router_weight);  // computed: only non-NULL matters
  aflex_status s = check_ffn(&f, true, true);
  if (s != AFLEX_OK) return s;
  REQUIRE(f.H <= 16384, AFLEX_ERR_UNSUPPORTED, "moe_block: H=%d above 16384", f.H);
  REQUIRE(aligned16(m->norm_weight) && aligned16(m->router_weight), AFLEX_ERR_ALIGNMENT,
          "moe_block: weights must be 16-byte aligned");
  return AFLEX_OK;
}

aflex_status aflex_moe_block_workspace(const aflex_moe_block_args* m, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "moe_block: bytes is NULL");
  aflex_status s = check_moe_block(m);
  if (s != AFLEX_OK) return s;
  *bytes = aflex::moe_block_workspace_bytes(*m);
  return AFLEX_OK;
}

aflex_status aflex_moe_block(const aflex_moe_block_args* m, void* ws, size_t ws_bytes, aflex_stream stream) {
  aflex_status s = check_moe_block(m);
  if (s != AFLEX_OK) return s;
  s = check_ws(ws, ws_bytes, aflex::moe_block_workspace_bytes(*m), "moe_block");
  if (s != AFLEX_OK) return s;
  return hip_status(aflex::launch_moe_block(*m, ws, (hipStream_t)stream), "moe_block");
}

aflex_status aflex_af_pipeline_workspace(const aflex_attn_args* a, const aflex_ffn_args* f, int32_t M,
                                         const int32_t* mb, int32_t L, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "pipeline: bytes is NULL");
  aflex_status s = check_pipe(a, f, M, mb, L);
  if (s != AFLEX_OK) return s;
  *bytes = pipe_layout(*a, *f, M, mb).total;
  return AFLEX_OK;
}

aflex_status aflex_af_pipeline_step(const aflex_attn_args* a, const aflex_ffn_args* f, int32_t M,
                                    const int32_t* mb, int32_t L, void* ws, size_t ws_bytes,
                                    aflex_stream stream_a, aflex_stream stream_f) {
  aflex_status s = check_pipe(a, f, M, mb, L);
  if (s != AFLEX_OK) return s;
  const PipeLayout P = pipe_layout(*a, *f, M, mb);
  s = check_ws(ws, ws_bytes, P.total, "pipeline");
  if (s != AFLEX_OK) return s;
  REQUIRE(stream_a != stream_f, AFLEX_ERR_INVALID_ARG, "pipeline: stream_a and stream_f must differ");

  hipStream_t sa = (hipStream_t)stream_a, sf = (hipStream_t)stream_f;
  char* w = static_cast<char*>(ws);
  uint16_t* attn_out = reinterpret_cast<uint16_t*>(w + P.attn_out);
  void* attn_ws = w + P.attn_ws;
  void* ffn_ws = w + P.ffn_ws;
  const int H = f->H;

  hipError_t e;
  std::lock_guard<std::mutex> lock(g_events.mu);
  std::vector<hipEvent_t>* evp = nullptr;
  s = pipeline_events(2 * (size_t)M + 1, &evp);
  if (s != AFLEX_OK) return s;
  std::vector<hipEvent_t>& ev = *evp;
  hipEvent_t entry = ev[0];
  hipEvent_t* evA = &ev[1];
  hipEvent_t* evF = &ev[1 + M];

  // Work still queued on stream_f from an earlier call may read the buffers
  // the first attention overwrites.
  if ((e = hipEventRecord(entry, sf)) != hipSuccess) return hip_status(e, "pipeline");
  if ((e = hipStreamWaitEvent(sa, entry, 0)) != hipSuccess) return hip_status(e, "pipeline");

  // Routing depends only on the router logits: do it for every microbatch up
  // front on stream_f, where it overlaps the first attention.
  if (f->E) {
    int off = 0;
    for (int i = 0; i < M; ++i) {
      aflex_ffn_args fm = mb_ffn(*f, off, mb[i]);
      if ((e = aflex::launch_moe_route(fm, w + P.route_ws + (size_t)i * P.route_stride, sf)) != hipSuccess)
        return hip_status(e, "pipeline: route");
      off += mb[i];
    }
  }

  for (int l = 0; l < L; ++l) {
    int off = 0;
    for (int i = 0; i < M; ++i) {
      const int n = mb[i];
      if (l > 0 && (e = hipStreamWaitEvent(sa, evF[i], 0)) != hipSuccess) return hip_status(e, "pipeline");
      aflex_attn_args am = mb_attn(*a, off, n);
      if (l > 0) am.q = f->y + (size_t)off * H;
      am.out = attn_out + (size_t)off * H;
      if ((e = aflex::launch_attn_decode(am, attn_ws, sa, aflex::AttnForm::kWide)) != hipSuccess)
        return hip_status(e, "pipeline: attn");
      if ((e = hipEventRecord(evA[i], sa)) != hipSuccess) return hip_status(e, "pipeline");
      if ((e = hipStreamWaitEvent(sf, evA[i], 0)) != hipSuccess) return hip_status(e, "pipeline");
      aflex_ffn_args fm = mb_ffn(*f, off, n);
      fm.x = attn_out + (size_t)off * H;
      e = f->E ? aflex::launch_moe_experts(fm, w + P.route_ws + (size_t)i * P.route_stride, ffn_ws, sf)
               : aflex::launch_swiglu(fm, ffn_ws, sf);
      if (e != hipSuccess) return hip_status(e, "pipeline: ffn");
      if ((e = hipEventRecord(evF[i], sf)) != hipSuccess) return hip_status(e, "pipeline");
      off += n;
    }
  }
  return AFLEX_OK;
}

aflex_status aflex_af_layer_workspace(const aflex_attn_args* a, const aflex_ffn_args* f, const aflex_layer_args* ly,
                                      int32_t M, const int32_t* mb, int32_t L, size_t* bytes) {
  REQUIRE(bytes, AFLEX_ERR_INVALID_ARG, "layer: bytes is NULL");
  aflex_status s = check_layer(a, f, ly, M, mb, L);
  if (s != AFLEX_OK) return s;
  *bytes = layer_layout(*a, *f, *ly, M, mb).total;
  return AFLEX_OK;
}

aflex_status aflex_af_layer_step(const aflex_attn_args* a, const aflex_ffn_args* f, const aflex_layer_args* ly,
                                 int32_t M, const int32_t* mb, int32_t L, void* ws, size_t ws_bytes,
                                 aflex_stream stream_a, aflex_stream stream_f) {
  aflex_status s = check_layer(a, f, ly, M, mb, L);
  if (s != AFLEX_OK) return s;
  const LayerLayout P = layer_layout(*a, *f, *ly, M, mb);
  s = check_ws(ws, ws_bytes, P.total, "layer");
  if (s != AFLEX_OK) return s;
  REQUIRE(stream_a != stream_f, AFLEX_ERR_INVALID_ARG, "layer: stream_a and stream_f must differ");

  hipStream_t sa = (hipStream_t)stream_a, sf = (hipStream_t)stream_f;
  char* w = static_cast<char*>(ws);
  uint16_t* attn_out = reinterpret_cast<uint16_t*>(w + P.attn_out);
  uint16_t* h = reinterpret_cast<uint16_t*>(w + P.h);
  const int H = f->H, HqD = a->Hq * a->D, kvrow = a->Hkv * a->D;

  hipError_t e;
  std::lock_guard<std::mutex> lock(g_events.mu);
  std::vector<hipEvent_t>* evp = nullptr;
  s = pipeline_events(2 * (size_t)M + 1, &evp);
  if (s != AFLEX_OK) return s;
  std::vector<hipEvent_t>& ev = *evp;
  hipEvent_t entry = ev[0];
  hipEvent_t* evA = &ev[1];
  hipEvent_t* evF = &ev[1 + M];

  // Work still queued on stream_f from an earlier call may read the buffers
  // the first attention stage overwrites.
  if ((e = hipEventRecord(entry, sf)) != hipSuccess) return hip_status(e, "layer");
  if ((e = hipStreamWaitEvent(sa, entry, 0)) != hipSuccess) return hip_status(e, "layer");

  for (int l = 0; l < L; ++l) {
    int off = 0;
    for (int i = 0; i < M; ++i) {
      const int n = mb[i];
      if (l > 0 && (e = hipStreamWaitEvent(sa, evF[i], 0)) != hipSuccess) return hip_status(e, "layer");
      // attention stage: append, attention, projection (+ the layer input)
      aflex_kv_append_args ka;
      ka.k_new = ly->k_new + (size_t)off * kvrow;
      ka.v_new = ly->v_new + (size_t)off * kvrow;
      ka.k_cache = ly->k_cache;
      ka.v_cache = ly->v_cache;
      ka.block_table = a->block_table + (size_t)off * a->max_blocks_per_seq;
      ka.context_lens = a->context_lens + off;
      ka.B = n;
      ka.Hkv = a->Hkv;
      ka.D = a->D;
      ka.block_size = a->block_size;
      ka.max_blocks_per_seq = a->max_blocks_per_seq;
      ka.num_blocks = a->num_blocks;
      if ((e = aflex::launch_kv_append(ka, sa)) != hipSuccess) return hip_status(e, "layer: kv append");
      aflex_attn_args am = mb_attn(*a, off, n);
      if (l > 0) am.q = f->y + (size_t)off * H;
      am.out = attn_out + (size_t)off * HqD;
      // The 4-wave form here: the attention stream also runs o_proj, which
      // shares the CUs better with it than with one 12-wave work-group per CU.
      if ((e = aflex::launch_attn_decode(am, w + P.attn_ws, sa, aflex::AttnForm::kShared)) != hipSuccess)
        return hip_status(e, "layer: attn");
      const uint16_t* res = l > 0 ? f->y + (size_t)off * H : (ly->x_in ? ly->x_in + (size_t)off * H : nullptr);
      const aflex_linear_args lin = mb_linear(*a, *f, *ly, am.out, h + (size_t)off * H, n);
      if ((e = aflex::launch_linear(lin, w + P.lin_ws, sa, res)) != hipSuccess) return hip_status(e, "layer: o_proj");
      if ((e = hipEventRecord(evA[i], sa)) != hipSuccess) return hip_status(e, "layer");
      // FFN stage: the MoE block on the hidden state that crossed the boundary
      if ((e = hipStreamWaitEvent(sf, evA[i], 0)) != hipSuccess) return hip_status(e, "layer");
      const aflex_moe_block_args blk = mb_block(*f, *ly, off, n, h + (size_t)off * H);
      if ((e = aflex::launch_moe_block(blk, w + P.blk_ws, sf)) != hipSuccess) return hip_status(e, "layer: moe block");
      if ((e = hipEventRecord(evF[i], sf)) != hipSuccess) return hip_status(e, "layer");
      off += n;
    }
  }
  return AFLEX_OK;
}

}  // extern "C"
