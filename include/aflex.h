/*
 * aflex.h -- C ABI of the decode-step Attention / FFN operator library for
 * AMD Instinct MI355X (gfx950).
 *
 * The paper (AFlex, "Energy-Efficient LLM Serving via Disaggregated
 * Attention-FFN and Flexible Frequency Scaling") disaggregates each decode
 * layer into an Attention stage (DA) and an FFN stage (DF) that exchange the
 * hidden states [tokens, hidden] at every layer boundary (section 4.3, "AFD
 * Data Plane") and runs them as an interleaved microbatch pipeline whose
 * timing Eq. 2 models. This library provides the two operators and that
 * pipeline on one GPU:
 *
 *   aflex_attn_decode       batched GQA decode attention over a paged KV cache
 *   aflex_attn_decode_noalloc  the same without a workspace (static scratch)
 *   aflex_ffn_swiglu        dense SwiGLU FFN (Qwen3-32B-shaped layers)
 *   aflex_moe_ffn           top-k mixture-of-experts SwiGLU FFN (Mixtral-8x7B)
 *   aflex_moe_block         RMSNorm + router + MoE FFN (+ residual)
 *   aflex_af_pipeline_step  M microbatches of A then F on two HIP streams
 *   aflex_af_layer_step     the same over a whole decode layer (KV append,
 *                           attention, output projection | MoE block)
 *   aflex_kv_append         the new token's K/V into the paged cache
 *   aflex_kv_write          a packed prompt's (or chunk's) K/V into the cache
 *   aflex_linear            y = x W^T (the attention output projection)
 *   aflex_attn_prefill      causal attention over packed prompts (prefill)
 *   aflex_pool_streams_*    stream pairs on disjoint CU sets (A/F pools)
 *   aflex_profile_*         per-kernel HIP-event timing
 *   aflex_teardown          release the HIP events the library caches
 *
 * Conventions shared by every entry point
 *  - bf16 tensors are passed as raw bit patterns (aflex_bf16 = uint16_t).
 *  - All tensor pointers are DEVICE pointers owned by the caller, dense
 *    row-major in the layout stated, 16-byte aligned. Inputs are read-only;
 *    outputs must not alias inputs.
 *  - Every call is asynchronous on the given stream(s) (an aflex_stream is a
 *    hipStream_t; NULL is the null stream). Nothing on the hot path allocates
 *    or synchronises with the host; the caller passes a device workspace of at
 *    least the size the matching *_workspace query returns, 256-byte aligned.
 *  - Arguments are validated on the host before anything is launched. On a
 *    non-OK status nothing has been launched and aflex_last_error() returns a
 *    message. Values that live in device memory (context lengths, block ids,
 *    logits) cannot be validated on the host; the kernels clamp them so that
 *    no access leaves the caller's buffers (see each entry point).
 *  - No function throws or aborts; HIP failures return AFLEX_ERR_HIP.
 */
#ifndef AFLEX_H
#define AFLEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t aflex_bf16;
typedef void *aflex_stream;

typedef enum aflex_status {
  AFLEX_OK = 0,
  AFLEX_ERR_INVALID_ARG = 1, /* null pointer, non-positive or inconsistent size */
  AFLEX_ERR_UNSUPPORTED = 2, /* a shape outside what the kernels implement */
  AFLEX_ERR_ALIGNMENT = 3,   /* a pointer that is not 16-byte aligned */
  AFLEX_ERR_WORKSPACE = 4,   /* workspace missing or smaller than required */
  AFLEX_ERR_HIP = 5          /* a HIP runtime call failed (message has details) */
} aflex_status;

/* ------------------------------------------------------------------------ */
/* Decode attention (DA). The decode step's attention reads the whole cached  */
/* context of every sequence (section 1; section 2, "LLM Serving"). For each  */
/* sequence b < B and query head h < Hq, with G = Hq / Hkv and g = h / G:     */
/*   k_j = k_cache[block_table[b][j / bs]][g][j % bs][:]      j < ctx_b       */
/*   v_j = v_cache[block_table[b][j / bs]][g][:][j % bs]                      */
/*   out[b][h] = sum_j softmax_j(scale * <q[b][h], k_j>) * v_j   (bf16)       */
/* ------------------------------------------------------------------------ */
typedef struct aflex_attn_args {
  const aflex_bf16 *q;         /* [B, Hq, D] */
  const aflex_bf16 *k_cache;   /* [num_blocks, Hkv, block_size, D] */
  const aflex_bf16 *v_cache;   /* [num_blocks, Hkv, D, block_size]  (token fastest) */
  const int32_t *block_table;  /* [B, max_blocks_per_seq]; entries >= ceil(ctx/bs) unread */
  const int32_t *context_lens; /* [B]; valid cached tokens incl. the current one */
  aflex_bf16 *out;             /* [B, Hq, D] */
  int32_t B, Hq, Hkv, D;
  int32_t block_size;          /* must be 16 */
  int32_t max_blocks_per_seq;  /* row stride of block_table */
  int32_t num_blocks;          /* blocks in each pool; ids outside [0, num_blocks) are skipped */
  int32_t max_context_len;     /* host-known bound on every ctx_b (<= max_blocks_per_seq*bs);
                                  sizes the launch grid, larger device values are clamped */
  float scale;                 /* softmax scale; 0 selects 1/sqrt(D) */
  int32_t split_tokens;        /* 0: the cached blocks of all (sequence, kv head) pairs are
                                  spread evenly over the work-groups the GPU holds at once;
                                  else each work-group takes this many tokens' blocks of them
                                  (a multiple of 128 in [128, 1024]) */
} aflex_attn_args;

/* Supported: D in {64, 128}, block_size == 16, Hkv >= 1, Hq % Hkv == 0,
 * 1 <= Hq / Hkv <= 16, B * Hkv * ceil(max_context_len / 16) < 2^30.
 * ctx_b == 0 yields out = 0. Block ids outside [0, num_blocks) contribute
 * nothing (their tokens are masked). Two launches on the stream: the split
 * attention, then a merge of the (sequence, kv head) pairs it split between
 * work-groups; the workspace holds their fp32 partials and needs no
 * initialisation. With split_tokens = 0, max_context_len <= 512 and B * Hkv
 * at most the resident work-groups, each pair takes one work-group whole and
 * the merge launch is skipped. The output is the same on every call with the
 * same inputs (bitwise). */
aflex_status aflex_attn_decode_workspace(const aflex_attn_args *a, size_t *bytes);
aflex_status aflex_attn_decode(const aflex_attn_args *a, void *workspace, size_t workspace_bytes,
                               aflex_stream stream);

/* Decode attention that allocates nothing, for callers that cannot call      */
/* hipMalloc or hand over a workspace: code under HIP graph capture, tight    */
/* serving loops, harnesses that forbid allocation. Same operation,           */
/* arguments, validation and result as aflex_attn_decode (the same kernels);  */
/* its split partials live in a static device array of the library, 64 MiB    */
/* per device (held from the library's load on that device until the process  */
/* ends). Shapes whose partials need more (the aflex_attn_decode_workspace    */
/* size, about (B * Hkv + 768) * (Hq / Hkv) * (D + 2) * 4 bytes on a 256-CU   */
/* device with split_tokens = 0) return AFLEX_ERR_WORKSPACE before anything   */
/* is launched. Every call on a device shares that device's array: calls that */
/* may overlap on one device (different streams without ordering, several     */
/* host threads) race and give wrong results; order them on one stream. No    */
/* HIP allocation, memset or host synchronisation happens in the call; the    */
/* first call on a device looks up the array's device address                 */
/* (hipGetSymbolAddress) once.                                                */
aflex_status aflex_attn_decode_noalloc(const aflex_attn_args *a, aflex_stream stream);

/* ------------------------------------------------------------------------ */
/* FFN (DF). Dense SwiGLU, the FFN of the dense model the paper evaluates     */
/* (Qwen3-32B, section 6.1), memory-bound at small decode batches and         */
/* compute-bound at large ones (section 1):                                   */
/*   y = (SiLU(x W_g^T) * (x W_u^T)) W_d^T,   SiLU(z) = z / (1 + exp(-z))    */
/* MoE: top-k of E SwiGLU experts (Mixtral-8x7B, section 6.1, section 6.2),   */
/*   ids_t = top-k experts by router logit (ties -> lower id),                */
/*   w_t   = softmax over the k selected logits,                              */
/*   y_t   = sum_j w_t,j * SwiGLU_{ids_t,j}(x_t).                             */
/* ------------------------------------------------------------------------ */
typedef struct aflex_ffn_args {
  const aflex_bf16 *x;          /* [T, H] */
  const float *router_logits;   /* [T, E] fp32 (MoE only; must be finite) */
  const aflex_bf16 *w_gate;     /* dense [I, H]; MoE [E, I, H] */
  const aflex_bf16 *w_up;       /* dense [I, H]; MoE [E, I, H] */
  const aflex_bf16 *w_down;     /* dense [H, I]; MoE [E, H, I] */
  aflex_bf16 *y;                /* [T, H] */
  int32_t *topk_ids;            /* MoE optional output [T, k] (NULL: not written) */
  float *topk_w;                /* MoE optional output [T, k] */
  int32_t *expert_offsets;      /* MoE optional output [E + 1]: exclusive prefix of counts */
  int32_t *sorted_pairs;        /* MoE optional output [T * k]: pair ids t*k+j ordered by
                                   (expert, token, slot) */
  int32_t T, H, I;
  int32_t E, k;                 /* MoE only: experts and experts per token (ignored by dense) */
} aflex_ffn_args;

/* Supported: H and I multiples of 64, T >= 1; MoE 1 <= k <= E <= 64, k <= 8. */
aflex_status aflex_ffn_swiglu_workspace(const aflex_ffn_args *f, size_t *bytes);
aflex_status aflex_ffn_swiglu(const aflex_ffn_args *f, void *workspace, size_t workspace_bytes,
                              aflex_stream stream);
aflex_status aflex_moe_ffn_workspace(const aflex_ffn_args *f, size_t *bytes);
aflex_status aflex_moe_ffn(const aflex_ffn_args *f, void *workspace, size_t workspace_bytes,
                           aflex_stream stream);

/* MoE FFN block of a Mixtral layer: the normalisation and router that come   */
/* before the experts (section 6.1 names the model):                         */
/*   xn     = x / sqrt(mean(x^2) + eps) * norm_weight        (per token)     */
/*   logits = xn W_r^T  (fp32, from the unrounded xn)        W_r = [E, H]    */
/*   y      = MoE(bf16(xn), logits)  (+ x when residual != 0)                */
/* ffn.x is the block input; ffn.router_logits is ignored (computed); the    */
/* optional MoE outputs of ffn are written as by aflex_moe_ffn.              */
typedef struct aflex_moe_block_args {
  aflex_ffn_args ffn;              /* MoE weights and shapes, ffn.x = input [T, H] */
  const aflex_bf16 *norm_weight;   /* [H] RMSNorm gain */
  const aflex_bf16 *router_weight; /* [E, H] */
  float eps;                       /* RMSNorm epsilon (>= 0) */
  int32_t residual;                /* nonzero: add x to the output */
  float *router_logits_out;        /* optional [T, E] fp32 output (NULL: not written) */
} aflex_moe_block_args;

/* Supported: as aflex_moe_ffn, and H <= 16384. */
aflex_status aflex_moe_block_workspace(const aflex_moe_block_args *m, size_t *bytes);
aflex_status aflex_moe_block(const aflex_moe_block_args *m, void *workspace, size_t workspace_bytes,
                             aflex_stream stream);

/* ------------------------------------------------------------------------ */
/* Interleaved A/F layer step (section 4.3, "Interleaved A/F Pipeline"; Eq. 2)*/
/* The batch is cut into M contiguous microbatches of host-known sizes        */
/* mb_sizes[0..M) (sum = B). Attention of microbatch i runs on stream_a, its  */
/* FFN on stream_f once that attention is done; A of layer step l+1 for       */
/* microbatch i starts as soon as F of step l for i is done, so A of one      */
/* microbatch overlaps F of another. The FFN input is the attention output    */
/* viewed as [n_i, Hq*D] (so ffn->H must equal Hq*D); for L > 1 the FFN       */
/* output viewed as [n_i, Hq, D] is the next step's q. ffn->E == 0 selects    */
/* the dense SwiGLU, else the MoE with router logits rows of microbatch i.    */
/* attn->q is the first step's q, attn->out is unused (may be NULL),          */
/* ffn->x is unused (may be NULL), ffn->y [B, H] receives the last step's     */
/* output and the optional MoE outputs are not written. On return stream_f    */
/* is ordered after all of the step's work on both streams.                   */
/* ------------------------------------------------------------------------ */
aflex_status aflex_af_pipeline_workspace(const aflex_attn_args *attn, const aflex_ffn_args *ffn,
                                         int32_t M, const int32_t *mb_sizes, int32_t L,
                                         size_t *bytes);
aflex_status aflex_af_pipeline_step(const aflex_attn_args *attn, const aflex_ffn_args *ffn,
                                    int32_t M, const int32_t *mb_sizes, int32_t L,
                                    void *workspace, size_t workspace_bytes,
                                    aflex_stream stream_a, aflex_stream stream_f);

/* ------------------------------------------------------------------------ */
/* The whole decode layer on the interleaved A/F step (section 4.3: the       */
/* attention group runs attention and sends its output to the FFN group,    */
/* which runs the FFN block; Eq. 2 times the two stages). For microbatch i:  */
/*   stream_a: append the new token's K/V (aflex_kv_append), attention,     */
/*             h_i = x_i + attn_i W_o^T     (x_i: the layer input rows of i, */
/*                                           or nothing when x_in is NULL)  */
/*   stream_f: y_i = h_i + MoE(RMSNorm(h_i), RMSNorm(h_i) W_r^T)            */
/*             (aflex_moe_block with the residual)                           */
/* h_i [n_i, H] bf16 is the tensor that crosses the A/F boundary. For L > 1 */
/* step l + 1 of microbatch i takes q = y_i viewed [n_i, Hq, D] and x = y_i  */
/* (so H must equal Hq * D), appends the same K/V again (the same slot, the */
/* same values) and starts once F of step l for i is done. attn->out is     */
/* unused; moe->x and moe->router_logits are unused (may be NULL); moe->y   */
/* [B, H] receives the last step's output; moe->E >= 1 (the MoE block).     */
/* ------------------------------------------------------------------------ */
typedef struct aflex_layer_args {
  const aflex_bf16 *k_new;          /* [B, Hkv, D] new token's key per sequence */
  const aflex_bf16 *v_new;          /* [B, Hkv, D] new token's value */
  aflex_bf16 *k_cache;              /* the pools attn->k_cache / attn->v_cache point at */
  aflex_bf16 *v_cache;              /*   (written by the append; must be the same pointers) */
  const aflex_bf16 *w_o;            /* [H, Hq * D] output projection */
  const aflex_bf16 *x_in;           /* [B, H] layer input added to the projection, or NULL */
  const aflex_bf16 *norm_weight;    /* [H] RMSNorm gain of the MoE block */
  const aflex_bf16 *router_weight;  /* [E, H] */
  float eps;                        /* RMSNorm epsilon (>= 0) */
} aflex_layer_args;

/* Supported: as aflex_attn_decode, aflex_linear, aflex_moe_block and        */
/* aflex_af_pipeline_step; H <= 16384. Errors as those entry points.         */
aflex_status aflex_af_layer_workspace(const aflex_attn_args *attn, const aflex_ffn_args *moe,
                                      const aflex_layer_args *layer, int32_t M, const int32_t *mb_sizes,
                                      int32_t L, size_t *bytes);
aflex_status aflex_af_layer_step(const aflex_attn_args *attn, const aflex_ffn_args *moe,
                                 const aflex_layer_args *layer, int32_t M, const int32_t *mb_sizes, int32_t L,
                                 void *workspace, size_t workspace_bytes, aflex_stream stream_a,
                                 aflex_stream stream_f);

/* ------------------------------------------------------------------------ */
/* Steps either side of decode attention in the attention stage.            */
/* KV append: each decode step adds the new token's key and value to the    */
/* growing cache before attention reads it (section 1; section 2). With the */
/* new token counted in context_lens, it is written at j = ctx_b - 1:        */
/*   k_cache[block_table[b][j / 16]][g][j % 16][:] = k_new[b][g][:]          */
/*   v_cache[block_table[b][j / 16]][g][:][j % 16] = v_new[b][g][:]          */
/* Nothing is written for ctx_b <= 0, for j beyond the table's capacity or   */
/* for block ids outside [0, num_blocks). Pools are updated in place.        */
/* ------------------------------------------------------------------------ */
typedef struct aflex_kv_append_args {
  const aflex_bf16 *k_new;     /* [B, Hkv, D] */
  const aflex_bf16 *v_new;     /* [B, Hkv, D] */
  aflex_bf16 *k_cache;         /* [num_blocks, Hkv, block_size, D] (written) */
  aflex_bf16 *v_cache;         /* [num_blocks, Hkv, D, block_size] (written) */
  const int32_t *block_table;  /* [B, max_blocks_per_seq] */
  const int32_t *context_lens; /* [B], including the new token */
  int32_t B, Hkv, D;
  int32_t block_size;          /* must be 16 */
  int32_t max_blocks_per_seq, num_blocks;
} aflex_kv_append_args;

/* Supported: D in {64, 128}, block_size == 16. No workspace. */
aflex_status aflex_kv_append(const aflex_kv_append_args *a, aflex_stream stream);

/* Packed multi-token KV-cache write: prefill populates the cache with the     */
/* prompt's keys and values (section 2, "LLM Serving"), and chunked prefill    */
/* appends a chunk. Sequence b's new tokens are rows cu_seqlens[b] ..          */
/* cu_seqlens[b+1]-1 of k_new / v_new and are the newest n_b cached tokens:    */
/* token i goes to position context_lens[b] - n_b + i (positions below 0 are   */
/* skipped). With one token per sequence this is aflex_kv_append.             */
typedef struct aflex_kv_write_args {
  const aflex_bf16 *k_new;     /* [T, Hkv, D] */
  const aflex_bf16 *v_new;     /* [T, Hkv, D] */
  const int32_t *cu_seqlens;   /* [B+1] device, nondecreasing, cu[0] = 0, cu[B] = T */
  aflex_bf16 *k_cache;         /* [num_blocks, Hkv, block_size, D] (written) */
  aflex_bf16 *v_cache;         /* [num_blocks, Hkv, D, block_size] (written) */
  const int32_t *block_table;  /* [B, max_blocks_per_seq] */
  const int32_t *context_lens; /* [B], cached tokens after the write */
  int32_t B, T, Hkv, D;
  int32_t max_seqlen;          /* host-known bound on n_b; sizes the grid */
  int32_t block_size;          /* must be 16 */
  int32_t max_blocks_per_seq, num_blocks;
} aflex_kv_write_args;

/* Supported: D in {64, 128}, block_size == 16, Hkv * D / 8 <= 1024,          */
/* B <= 65535. No workspace. Device-side values are clamped: prompts to       */
/* [0, T], sequences with context_lens outside [1, capacity] and block ids    */
/* outside [0, num_blocks) write nothing; tokens of a sequence longer than    */
/* max_seqlen beyond the grid's reach are not written.                         */
aflex_status aflex_kv_write(const aflex_kv_write_args *a, aflex_stream stream);

/* Linear layer y = x W^T in bf16 with fp32 accumulation: the output           */
/* projection that brings the attention output back to the hidden size        */
/* before it crosses the A/F boundary (section 4.3).                           */
typedef struct aflex_linear_args {
  const aflex_bf16 *x;  /* [T, K] */
  const aflex_bf16 *w;  /* [N, K] (out_features, in_features) */
  aflex_bf16 *y;        /* [T, N] */
  int32_t T, K, N;      /* K and N multiples of 64 */
} aflex_linear_args;

aflex_status aflex_linear_workspace(const aflex_linear_args *l, size_t *bytes);
aflex_status aflex_linear(const aflex_linear_args *l, void *workspace, size_t workspace_bytes,
                          aflex_stream stream);

/* Causal prefill attention (section 2, "LLM Serving": prefill processes the  */
/* prompt tokens in parallel; section 3.2 profiles prefill Attention, PA,     */
/* next to decode). Prompts are packed back to back: prompt b is tokens       */
/* cu_seqlens[b] .. cu_seqlens[b+1]-1 of q, k, v. For token i of prompt b and */
/* query head h (g = h / (Hq/Hkv)):                                           */
/*   out[cu_b+i, h] = sum_{j<=i} softmax_j(scale <q[cu_b+i,h], k[cu_b+j,g]>)  */
/*                    v[cu_b+j, g]                                            */
/* bf16 in, fp32 accumulation, bf16 out (round to nearest even).              */
typedef struct aflex_prefill_args {
  const aflex_bf16 *q;          /* [T, Hq, D] */
  const aflex_bf16 *k;          /* [T, Hkv, D] */
  const aflex_bf16 *v;          /* [T, Hkv, D] */
  const int32_t *cu_seqlens;    /* [B+1] device, 0 = cu[0] <= cu[1] <= ... <= cu[B] = T */
  aflex_bf16 *out;              /* [T, Hq, D] */
  int32_t B, T, Hq, Hkv, D;
  int32_t max_seqlen;           /* host-known bound on every prompt length; sizes the grid and
                                   selects the work-group shape (two query heads per
                                   work-group from 2048 on, for an even Hq / Hkv), so a
                                   tight bound keeps short prompts on the faster shape */
  float scale;                  /* softmax scale; 0 selects 1/sqrt(D) */
} aflex_prefill_args;

/* Supported: D == 128, Hq % Hkv == 0, B <= 65535. No workspace.               */
/* cu_seqlens lives in device memory and is not checked on the host: the      */
/* kernel clamps each prompt to [0, T], so a bad array cannot make it read or */
/* write outside q, k, v, out; rows of a prompt longer than max_seqlen past   */
/* position max_seqlen are not written. Empty prompts produce no rows.        */
aflex_status aflex_attn_prefill(const aflex_prefill_args *a, aflex_stream stream);

/* Two streams whose kernels run on disjoint sets of compute units: the       */
/* single-GPU analogue of the paper's separate Attention and FFN GPU pools    */
/* (section 4.1, section 4.3) for aflex_af_pipeline_step. attn_cus of the 256 */
/* CUs serve stream_a, the others stream_f; attn_cus must be 64, 128 or 192.  */
/* Each XCD gives the same share of its CUs to each pool (the masks take bit  */
/* i for the attention pool when (i / 8) % 4 < attn_cus / 64, which is even   */
/* per XCD whether CU bits are numbered XCD by XCD or interleaved across     */
/* XCDs). Streams have the default priority. The caller releases them with   */
/* aflex_pool_streams_destroy. Errors: INVALID_ARG for NULL outputs,          */
/* UNSUPPORTED for another attn_cus or a device without 256 CUs, HIP when     */
/* stream creation fails (nothing is left allocated then).                    */
aflex_status aflex_pool_streams_create(int32_t attn_cus, aflex_stream *stream_a, aflex_stream *stream_f);
aflex_status aflex_pool_streams_destroy(aflex_stream stream_a, aflex_stream stream_f);

/* ------------------------------------------------------------------------ */
/* Per-kernel timing, the single-GPU analogue of the paper's per-operator     */
/* latency profiling (section 4.1; section 5, "Profiling module"). Between    */
/* aflex_profile_start and aflex_profile_stop, every library kernel whose     */
/* name is in the comma-separated list `kernels` (NULL or "" = all) is        */
/* bracketed by two HIP events on the stream it is launched on. Kernel names: */
/* attn_decode, attn_merge, gemm_gate_up, gemm_down, splitk_reduce,          */
/* moe_route, moe_combine, kv_append, kv_write, rmsnorm_router, attn_prefill. */
/* aflex_profile_stop waits for those events and writes one line per kernel   */
/* into `report` (host buffer of `len` bytes, truncated to fit):              */
/*   <name> <launches> <total_ms> <min_ms> <max_ms>                           */
/* Off by default; while off no event is recorded.                            */
/* ------------------------------------------------------------------------ */
aflex_status aflex_profile_start(const char *kernels);
aflex_status aflex_profile_stop(char *report, size_t len);

/* Releases the HIP objects the library keeps between calls: the events that */
/* order the two streams of aflex_af_pipeline_step (per device) and the       */
/* timing events of aflex_profile_*. Call it before process exit (or before  */
/* unloading the library) once no library work is queued on any stream,      */
/* e.g. after hipDeviceSynchronize(); streams from aflex_pool_streams_create  */
/* are the caller's to destroy. The library stays usable: the next call      */
/* creates what it needs again. Errors: HIP if a destroy failed (the others  */
/* are still destroyed).                                                     */
aflex_status aflex_teardown(void);

/* Thread-local message describing the last non-OK status of this thread. */
const char *aflex_last_error(void);
/* Library version string. */
const char *aflex_version(void);

#ifdef __cplusplus
}
#endif
#endif /* AFLEX_H */
