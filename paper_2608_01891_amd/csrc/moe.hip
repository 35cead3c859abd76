// Top-k mixture-of-experts SwiGLU FFN, gfx950.
//
// The FFN of the MoE model the paper evaluates (Mixtral-8x7B, section 6.1;
// section 6.2 "Generality" notes that sparse expert execution changes the
// FFN's computation and communication). Steps, all on the device and without
// a host synchronisation:
//   1. route: per token, top-k experts by logit (ties -> lower id) and the
//      softmax over the k selected logits; per-expert counts, their exclusive
//      prefix, the stable (expert, token, slot) order of the token/slot pairs,
//      each pair's position in that order, and the m-tile map of the grouped
//      GEMMs. One work-group up to 512 tokens, else three kernels over chunks
//      of 256 tokens; ranks come from wave ballots, so the order is
//      deterministic (and the same for both paths).
//   2. grouped gate/up GEMM with fused SwiGLU; the A rows are gathered from x
//      through the pair order (no permuted copy of x is written).
//   3. grouped down GEMM into fp32 split-K partials, rows in pair order.
//   4. combine: y_t = sum_j w_t,j * (sum over splits of row pos(t,j)), fixed
//      order, bf16 out.
#include "ffn_plan.h"
#include "gemm.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

constexpr int kMaxK = 8;
constexpr int kMaxE = 64;
// Up to this many tokens one work-group routes the batch (a single launch);
// larger batches take three kernels that spread the tokens over work-groups.
constexpr int kSingleRouteMaxT = 512;

// Workspace: a routing block (ids .. num_tiles, written by the route kernel)
// followed by the expert block (h, P). The two can live apart: the pipeline
// keeps one routing block per microbatch and one shared expert block.
struct MoeLayout {
  size_t ids, wts, offsets, sorted, pos, tile_map, num_tiles, blockcnt, blockbase, route_total;
  size_t h, P, expert_total;
  int bm, max_tiles, down_splits, down_kps;
  // 64- and 128-row tiles: experts' rows are expected to fit one tile
  // (average rows per expert x 1.3 <= bm, the margin pick_bm uses for 32-row
  // tiles), so each expert's weights are streamed once and load
  // non-temporally (measured 4-5% faster at 32-48 rows per expert on 64-row
  // tiles, 11% at 64 rows per expert on 128-row tiles).
  bool once;
};

static MoeLayout moe_layout(const aflex_ffn_args& f) {
  MoeLayout L;
  const size_t pairs = (size_t)f.T * f.k;
  L.bm = pick_bm((double)pairs / f.E);
  L.once = (L.bm == 64 || L.bm == 128) && (double)pairs / f.E * 1.3 <= (double)L.bm;
  L.max_tiles = (int)((pairs + L.bm - 1) / L.bm) + f.E;
  const int ntiles = (f.H + down_bn(L.bm) - 1) / down_bn(L.bm);
  // The tile count is a worst case here (the routing stays on the device):
  // round filling only for the one-work-group-per-CU tiles, as measured.
  plan_splits(L.max_tiles * ntiles, f.I, down_target(L.bm), L.bm >= 128 ? concurrent_wgs(L.bm) : 0, 16,
              &L.down_splits, &L.down_kps);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o += align_up(bytes, 256);
    return at;
  };
  L.ids = take(pairs * 4);
  L.wts = take(pairs * 4);
  L.offsets = take((size_t)(f.E + 1) * 4);
  L.sorted = take(pairs * 4);
  L.pos = take(pairs * 4);
  L.tile_map = take((size_t)L.max_tiles * 3 * 4);
  L.num_tiles = take(4);
  const size_t nblk = ((size_t)f.T + 255) / 256;
  L.blockcnt = take(nblk * f.E * 4);
  L.blockbase = take(nblk * f.E * 4);
  L.route_total = o;
  o = 0;
  L.h = take(pairs * f.I * 2);
  L.P = take((size_t)L.down_splits * pairs * f.H * 4);
  L.expert_total = o;
  return L;
}

size_t moe_route_bytes(const aflex_ffn_args& f) { return moe_layout(f).route_total; }
size_t moe_expert_bytes(const aflex_ffn_args& f) { return moe_layout(f).expert_total; }
size_t moe_workspace_bytes(const aflex_ffn_args& f) {
  const MoeLayout L = moe_layout(f);
  return L.route_total + L.expert_total;
}

// Top-k of one token's logits (descending, ties to the lower id) and the
// softmax over the selected ones.
__device__ __forceinline__ void topk_token(const float* l, int E, int k, int* sid, float* w) {
  uint64_t taken = 0;
  float sel[kMaxK];
  for (int j = 0; j < k; ++j) {
    int bi = -1;
    float bv = 0.f;
    for (int e = 0; e < E; ++e) {
      if ((taken >> e) & 1) continue;
      const float v = l[e];
      if (bi < 0 || v > bv) {
        bi = e;
        bv = v;
      }
    }
    taken |= 1ull << bi;
    sel[j] = bv;
    sid[j] = bi;
  }
  float z = 0.f, ex[kMaxK];
  for (int j = 0; j < k; ++j) {
    ex[j] = expf(sel[j] - sel[0]);
    z += ex[j];
  }
  for (int j = 0; j < k; ++j) w[j] = ex[j] / z;
}

// Copy the logits of `rows` tokens (rows of E floats, contiguous) into LDS rows
// of stride ls, eight independent loads per lane in flight at a time: the
// top-k then reads LDS instead of issuing one dependent global load per
// compared logit (about 16 serial memory round trips per token at E = 8,
// k = 2).
__device__ __forceinline__ void stage_logits(const float* __restrict__ src, int rows, int E, int ls, float* s_log,
                                             int tid) {
  const int n = rows * E;
  for (int i0 = 0; i0 < n; i0 += 256 * 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 + tid;
      v[u] = i < n ? src[i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 + tid;
      if (i < n) {
        const int r = i / E;
        s_log[r * ls + (i - r * E)] = v[u];
      }
    }
  }
}

// m-tiles of bm rows per expert, in expert order (one thread).
__device__ __forceinline__ void build_tile_map(const int* off, int E, int bm, int32_t* tile_map, int32_t* num_tiles) {
  int nt = 0;
  for (int e = 0; e < E; ++e)
    for (int r = off[e]; r < off[e + 1]; r += bm) {
      tile_map[3 * nt + 0] = e;
      tile_map[3 * nt + 1] = r;
      tile_map[3 * nt + 2] = min(r + bm, off[e + 1]);
      ++nt;
    }
  *num_tiles = nt;
}

// Stable rank of each of a 256-token chunk's pairs among the chunk's pairs of
// the same expert (token order, i.e. wave by wave, lane by lane): pre[j] within
// the wave, wcnt[w][e] the pairs of expert e in wave w.
__device__ __forceinline__ void chunk_ranks(const int* my_e, bool valid, int E, int k, int wave, int lane, int* pre,
                                            int (*wcnt)[kMaxE]) {
  const uint64_t lt = (1ull << lane) - 1ull;
  uint64_t mask = 0;
  for (int j = 0; j < k; ++j) {
    pre[j] = 0;
    if (valid) mask |= 1ull << my_e[j];
  }
  for (int e = 0; e < E; ++e) {
    const bool f = (mask >> e) & 1ull;
    const uint64_t bal = __ballot(f);
    if (f) {
      const int pr = __popcll(bal & lt);
      for (int j = 0; j < k; ++j)
        if (my_e[j] == e) pre[j] = pr;
    }
    if (lane == 0) wcnt[wave][e] = __popcll(bal);
  }
}

__global__ __launch_bounds__(256) void moe_route_kernel(const float* __restrict__ logits, int T, int E, int k,
                                                        int bm, int32_t* ids, float* wts, int32_t* offsets,
                                                        int32_t* sorted, int32_t* pos, int32_t* tile_map,
                                                        int32_t* num_tiles, int32_t* u_ids, float* u_w,
                                                        int32_t* u_offsets, int32_t* u_sorted) {
  __shared__ int cnt[kMaxE];
  __shared__ int off[kMaxE + 1];
  __shared__ int base[kMaxE];
  __shared__ int wcnt[4][kMaxE];
  __shared__ float s_log[256 * (kMaxE + 1)];        // one chunk's logits, rows of odd stride
  __shared__ int s_ids[kSingleRouteMaxT * kMaxK];  // selected experts, read back by step 3
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int ls = E | 1;
  if (tid < kMaxE) {
    cnt[tid] = 0;
    base[tid] = 0;
  }
  __syncthreads();

  // 1. top-k and softmax over the selected logits, 256 tokens at a time.
  for (int c0 = 0; c0 < T; c0 += 256) {
    stage_logits(logits + (size_t)c0 * E, min(256, T - c0), E, ls, s_log, tid);
    __syncthreads();
    const int t = c0 + tid;
    if (t < T) {
      int sid[kMaxK];
      float w[kMaxK];
      topk_token(s_log + tid * ls, E, k, sid, w);
      for (int j = 0; j < k; ++j) {
        ids[t * k + j] = sid[j];
        wts[t * k + j] = w[j];
        s_ids[t * k + j] = sid[j];
        if (u_ids) u_ids[t * k + j] = sid[j];
        if (u_w) u_w[t * k + j] = w[j];
        atomicAdd(&cnt[sid[j]], 1);
      }
    }
    __syncthreads();
  }

  // 2. offsets and the m-tile map.
  if (tid == 0) {
    off[0] = 0;
    for (int e = 0; e < E; ++e) off[e + 1] = off[e] + cnt[e];
    build_tile_map(off, E, bm, tile_map, num_tiles);
  }
  __syncthreads();
  if (tid <= E) {
    offsets[tid] = off[tid];
    if (u_offsets) u_offsets[tid] = off[tid];
  }

  // 3. stable ranks: pairs of expert e are ordered by token (a token holds e
  //    at most once), chunk by chunk of 256 tokens, wave by wave, lane by lane.
  for (int c0 = 0; c0 < T; c0 += 256) {
    const int t = c0 + tid;
    const bool valid = t < T;
    int my_e[kMaxK], pre[kMaxK];
    for (int j = 0; j < k; ++j) my_e[j] = valid ? s_ids[t * k + j] : -1;
    chunk_ranks(my_e, valid, E, k, wave, lane, pre, wcnt);
    __syncthreads();
    if (valid) {
      for (int j = 0; j < k; ++j) {
        const int e = my_e[j];
        int r = base[e] + pre[j];
        for (int w = 0; w < wave; ++w) r += wcnt[w][e];
        const int pidx = off[e] + r;
        sorted[pidx] = t * k + j;
        pos[t * k + j] = pidx;
        if (u_sorted) u_sorted[pidx] = t * k + j;
      }
    }
    __syncthreads();
    if (tid < E) base[tid] += wcnt[0][tid] + wcnt[1][tid] + wcnt[2][tid] + wcnt[3][tid];
    __syncthreads();
  }
}

// The same routing for larger batches in three kernels, so that the per-token
// work is spread over one work-group per 256 tokens instead of looping in one:
// (1) top-k and the chunk's expert counts, (2) offsets, tile map and each
// chunk's first rank per expert, (3) the chunk's stable ranks. The pair order
// is the single kernel's.
__global__ __launch_bounds__(256) void moe_topk_kernel(const float* __restrict__ logits, int T, int E, int k,
                                                       int32_t* ids, float* wts, int32_t* u_ids, float* u_w,
                                                       int32_t* blockcnt) {
  __shared__ int cnt[kMaxE];
  __shared__ float s_log[256 * (kMaxE + 1)];
  const int tid = threadIdx.x;
  const int ls = E | 1;
  if (tid < kMaxE) cnt[tid] = 0;
  const int t0 = blockIdx.x * 256;
  stage_logits(logits + (size_t)t0 * E, min(256, T - t0), E, ls, s_log, tid);
  __syncthreads();
  const int t = t0 + tid;
  if (t < T) {
    int sid[kMaxK];
    float w[kMaxK];
    topk_token(s_log + tid * ls, E, k, sid, w);
    for (int j = 0; j < k; ++j) {
      ids[t * k + j] = sid[j];
      wts[t * k + j] = w[j];
      if (u_ids) u_ids[t * k + j] = sid[j];
      if (u_w) u_w[t * k + j] = w[j];
      atomicAdd(&cnt[sid[j]], 1);
    }
  }
  __syncthreads();
  if (tid < E) blockcnt[(size_t)blockIdx.x * E + tid] = cnt[tid];
}

__global__ __launch_bounds__(256) void moe_offsets_kernel(const int32_t* __restrict__ blockcnt, int nblk, int E,
                                                          int bm, int32_t* offsets, int32_t* u_offsets,
                                                          int32_t* tile_map, int32_t* num_tiles,
                                                          int32_t* blockbase) {
  __shared__ int tot[kMaxE];
  __shared__ int off[kMaxE + 1];
  const int tid = threadIdx.x;
  if (tid < E) {
    int sum = 0;
    for (int b = 0; b < nblk; ++b) {
      blockbase[(size_t)b * E + tid] = sum;
      sum += blockcnt[(size_t)b * E + tid];
    }
    tot[tid] = sum;
  }
  __syncthreads();
  if (tid == 0) {
    off[0] = 0;
    for (int e = 0; e < E; ++e) off[e + 1] = off[e] + tot[e];
    build_tile_map(off, E, bm, tile_map, num_tiles);
  }
  __syncthreads();
  if (tid <= E) {
    offsets[tid] = off[tid];
    if (u_offsets) u_offsets[tid] = off[tid];
  }
}

__global__ __launch_bounds__(256) void moe_rank_kernel(const int32_t* __restrict__ ids, int T, int E, int k,
                                                       const int32_t* __restrict__ offsets,
                                                       const int32_t* __restrict__ blockbase, int32_t* sorted,
                                                       int32_t* pos, int32_t* u_sorted) {
  __shared__ int wcnt[4][kMaxE];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int t = blockIdx.x * 256 + tid;
  const bool valid = t < T;
  int my_e[kMaxK], pre[kMaxK];
  for (int j = 0; j < k; ++j) my_e[j] = valid ? ids[t * k + j] : -1;
  chunk_ranks(my_e, valid, E, k, wave, lane, pre, wcnt);
  __syncthreads();
  if (valid) {
    for (int j = 0; j < k; ++j) {
      const int e = my_e[j];
      int r = blockbase[(size_t)blockIdx.x * E + e] + pre[j];
      for (int w = 0; w < wave; ++w) r += wcnt[w][e];
      const int pidx = offsets[e] + r;
      sorted[pidx] = t * k + j;
      pos[t * k + j] = pidx;
      if (u_sorted) u_sorted[pidx] = t * k + j;
    }
  }
}

// The loads are issued in two independent batches -- the token's pair
// positions and weights (and the routed tile count), then the partial rows of
// up to four splits for all k pairs -- so a token waits for two memory round
// trips instead of one per pair and per split (inside the two-stream step,
// where every round trip queues behind the attention stream's loads, the
// chained form took 44 us per 64-token call on average). Sums keep split order
// per pair, then pair order.
template <int KMAX>
__global__ __launch_bounds__(256) void moe_combine_kernel(const float* __restrict__ P, long long split_stride,
                                                          int splits, int split_slots,
                                                          const int32_t* __restrict__ num_tiles, int n_ntiles,
                                                          int ksteps, const int32_t* __restrict__ pos,
                                                          const float* __restrict__ w, int k, int H,
                                                          const uint16_t* __restrict__ residual,
                                                          uint16_t* __restrict__ y) {
  const int t = blockIdx.x;
  const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (c >= H) return;
  const int routed = split_slots > 0 ? *num_tiles : 0;
  long long row[KMAX];
  float wt[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {  // pairs past k re-read the last one and are not added
    const int jj = min(j, k - 1);
    row[j] = pos[t * k + jj];
    wt[j] = w[t * k + jj];
  }
  // Uses of the loaded values here keep the compiler from sinking these loads
  // below the split planning, which waits for the routed tile count: all of
  // them then share one round trip.
  asm volatile("" ::"s"(routed));
#pragma unroll
  for (int j = 0; j < KMAX; ++j) asm volatile("" ::"s"(row[j]), "s"(wt[j]));
  if (split_slots > 0) {  // the down GEMM planned its split count on the device
    int kps;
    split_plan_slots(routed * n_ntiles, ksteps, splits, split_slots, &splits, &kps);
  }
  // Splits past the last re-read it and are not added; sums start from -0,
  // which leaves the first split's value unchanged.
  constexpr int kBatch = 4;
  f32x4 s[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) s[j] = f32x4{-0.f, -0.f, -0.f, -0.f};
  for (int sp0 = 0; sp0 < splits; sp0 += kBatch) {
    f32x4 v[kBatch][KMAX];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        v[u][j] = *reinterpret_cast<const f32x4*>(P + min(sp0 + u, splits - 1) * split_stride + row[j] * H + c);
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        if (sp0 + u < splits) s[j] += v[u][j];
  }
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < KMAX; ++j)
    if (j < k) acc += wt[j] * s[j];
  if (residual) {
    const ushort4 rv = *reinterpret_cast<const ushort4*>(residual + (size_t)t * H + c);
    acc[0] += bf2f(rv.x);
    acc[1] += bf2f(rv.y);
    acc[2] += bf2f(rv.z);
    acc[3] += bf2f(rv.w);
  }
  ushort4 o;
  o.x = f2bf(acc[0]);
  o.y = f2bf(acc[1]);
  o.z = f2bf(acc[2]);
  o.w = f2bf(acc[3]);
  *reinterpret_cast<ushort4*>(y + (size_t)t * H + c) = o;
}

hipError_t launch_moe_route(const aflex_ffn_args& f, void* route_ws, hipStream_t stream) {
  const MoeLayout L = moe_layout(f);
  char* w = static_cast<char*>(route_ws);
  int32_t* ids = reinterpret_cast<int32_t*>(w + L.ids);
  float* wts = reinterpret_cast<float*>(w + L.wts);
  int32_t* offsets = reinterpret_cast<int32_t*>(w + L.offsets);
  int32_t* sorted = reinterpret_cast<int32_t*>(w + L.sorted);
  int32_t* pos = reinterpret_cast<int32_t*>(w + L.pos);
  int32_t* tile_map = reinterpret_cast<int32_t*>(w + L.tile_map);
  int32_t* num_tiles = reinterpret_cast<int32_t*>(w + L.num_tiles);
  ProfScope ps("moe_route", stream);
  if (f.T <= kSingleRouteMaxT) {
    moe_route_kernel<<<1, 256, 0, stream>>>(f.router_logits, f.T, f.E, f.k, L.bm, ids, wts, offsets, sorted, pos,
                                            tile_map, num_tiles, f.topk_ids, f.topk_w, f.expert_offsets,
                                            f.sorted_pairs);
    return hipGetLastError();
  }
  const int nblk = (f.T + 255) / 256;
  int32_t* blockcnt = reinterpret_cast<int32_t*>(w + L.blockcnt);
  int32_t* blockbase = reinterpret_cast<int32_t*>(w + L.blockbase);
  moe_topk_kernel<<<nblk, 256, 0, stream>>>(f.router_logits, f.T, f.E, f.k, ids, wts, f.topk_ids, f.topk_w,
                                            blockcnt);
  moe_offsets_kernel<<<1, 256, 0, stream>>>(blockcnt, nblk, f.E, L.bm, offsets, f.expert_offsets, tile_map,
                                            num_tiles, blockbase);
  moe_rank_kernel<<<nblk, 256, 0, stream>>>(ids, f.T, f.E, f.k, offsets, blockbase, sorted, pos,
                                            f.sorted_pairs);
  return hipGetLastError();
}

hipError_t launch_moe(const aflex_ffn_args& f, void* ws, hipStream_t stream, const uint16_t* residual) {
  const MoeLayout L = moe_layout(f);
  hipError_t e = launch_moe_route(f, ws, stream);
  if (e != hipSuccess) return e;
  return launch_moe_experts(f, ws, static_cast<char*>(ws) + L.route_total, stream, residual);
}

hipError_t launch_moe_experts(const aflex_ffn_args& f, void* route_ws, void* expert_ws, hipStream_t stream,
                              const uint16_t* residual) {
  const MoeLayout L = moe_layout(f);
  char* w = static_cast<char*>(route_ws);
  char* xw = static_cast<char*>(expert_ws);
  const float* wts = reinterpret_cast<const float*>(w + L.wts);
  const int32_t* sorted = reinterpret_cast<const int32_t*>(w + L.sorted);
  const int32_t* pos = reinterpret_cast<const int32_t*>(w + L.pos);
  const int32_t* tile_map = reinterpret_cast<const int32_t*>(w + L.tile_map);
  const int32_t* num_tiles = reinterpret_cast<const int32_t*>(w + L.num_tiles);
  uint16_t* h = reinterpret_cast<uint16_t*>(xw + L.h);
  float* P = reinterpret_cast<float*>(xw + L.P);
  hipError_t e;

  GemmParams g = {};
  g.A = f.x;
  g.lda = f.H;
  g.gather = sorted;
  g.gather_div = f.k;
  g.B0 = f.w_gate;
  g.B1 = f.w_up;
  g.ldb = f.H;
  g.b_expert_stride = (long long)f.I * f.H;
  g.N = f.I;
  g.K = f.H;
  g.k_per_split = f.H;
  g.splits = 1;
  g.tile_map = tile_map;
  g.num_mtiles = num_tiles;
  g.max_mtiles = L.max_tiles;
  g.n_ntiles = (f.I + gate_bn(L.bm) - 1) / gate_bn(L.bm);
  // Experts expected in one row tile each (their weights streamed once):
  // expert-major order over the device-side tile count, so each XCD takes
  // consecutive n-tiles of one or two experts and keeps their token rows in
  // its L2 (64 tokens: 452 -> 444 us; the down GEMM at 256 tokens 179 -> 174
  // us). Otherwise an expert's m-tiles stay adjacent, so its overflow tiles
  // re-read the weights from L2 (the expert-major order took 512 tokens from
  // 745 to 820 us).
  const int order = (L.bm == 32 || L.once) ? 2 : 0;
  g.mt_major = order;
  g.C = h;
  g.ldc = f.I;
  e = launch_gate_up(L.bm, L.once, g, stream);
  if (e != hipSuccess) return e;

  const long long pairs = (long long)f.T * f.k;
  GemmParams d = {};
  d.A = h;
  d.lda = f.I;
  d.B0 = f.w_down;
  d.ldb = f.I;
  d.b_expert_stride = (long long)f.H * f.I;
  d.N = f.H;
  d.K = f.I;
  d.k_per_split = L.down_kps;
  d.splits = L.down_splits;
  // One-work-group-per-CU tiles: the split count follows the routed tile
  // count (at most the worst-case plan's), so whole rounds stay filled
  // without fp32 partials the tile count does not need (2048 tokens: one
  // split instead of three).
  d.split_slots = L.bm >= 128 ? concurrent_wgs(L.bm) : 0;
  d.tile_map = tile_map;
  d.num_mtiles = num_tiles;
  d.max_mtiles = L.max_tiles;
  d.n_ntiles = (f.H + down_bn(L.bm) - 1) / down_bn(L.bm);
  d.mt_major = order;
  d.P = P;
  d.p_split_stride = pairs * f.H;
  d.ldp = f.H;
  e = launch_down(L.bm, true, L.once, d, stream);
  if (e != hipSuccess) return e;

  dim3 grid(f.T, (f.H / 4 + 255) / 256);
  ProfScope ps("moe_combine", stream);
  if (f.k <= 2)
    moe_combine_kernel<2><<<grid, 256, 0, stream>>>(P, d.p_split_stride, L.down_splits, d.split_slots, num_tiles,
                                                    d.n_ntiles, f.I / 64, pos, wts, f.k, f.H, residual, f.y);
  else
    moe_combine_kernel<kMaxK><<<grid, 256, 0, stream>>>(P, d.p_split_stride, L.down_splits, d.split_slots,
                                                        num_tiles, d.n_ntiles, f.I / 64, pos, wts, f.k, f.H,
                                                        residual, f.y);
  return hipGetLastError();
}

}  // namespace aflex
