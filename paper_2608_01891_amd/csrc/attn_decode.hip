// Batched GQA decode attention over a paged bf16 KV cache, gfx950.
//
// Operation: for every sequence b and query head h, softmax-weighted sum of
// the cached values of kv head g = h / G over the ctx_b cached tokens, the
// decode-step attention the paper treats as the memory-bound operator
// (section 1; section 3.2).
//
// Design (HBM-bound: every cached K/V byte is read exactly once):
//  * split kernel: one work-group of 4 waves per (sequence, kv head, split of
//    split_tokens tokens). Waves take pairs of 16-token blocks round-robin.
//    Per pair a wave issues 16 (D=128) 16-byte loads per lane straight into
//    MFMA operand registers -- no LDS staging is needed because both
//    contractions see their operand with the contraction index contiguous:
//      S^T[tok][g] = K[tok][:] . q[g][:]       (v_mfma_f32_16x16x32_bf16,
//                                               K rows = 16 tokens, 16 cols = G
//                                               query heads padded to 16)
//      O^T[d][g]  += V^T[d][tok] . P^T[tok][g]  (V pool is [.., D, 16] so 8
//                                               consecutive tokens of one d are
//                                               one 16-byte load)
//    The token order inside the QK tile is chosen so that the S^T output
//    registers of a lane are exactly the P^T operand registers it needs for
//    the PV product, and all softmax state of head g lives in the four lanes
//    with lane % 16 == g: the online softmax needs two cross-lane max steps per
//    block pair and no LDS round trip.
//  * the 4 waves of a work-group merge through LDS; a sequence with a single
//    split writes bf16 output directly, longer ones write an fp32 partial
//    (O, m, l) for the merge kernel.
//  * merge kernel: one wave per (sequence, head) rescales and sums the splits.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

struct AttnParams {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* bt;
  const int32_t* cl;
  uint16_t* out;
  float* part_o;   // [B*Hq, max_splits, D]
  float* part_ml;  // [B*Hq, max_splits, 2]  (running max in log2 units, sum)
  int B, Hq, Hkv, G;
  int max_blocks, num_blocks, max_ctx;
  int split_tokens, max_splits;
  float scale_log2;  // softmax scale * log2(e)
};

constexpr int kWaves = 4;

__device__ __forceinline__ int clamp_ctx(const AttnParams& p, int b) {
  int c = p.cl[b];
  return c < 0 ? 0 : (c > p.max_ctx ? p.max_ctx : c);
}

// K/V tile loads; NT marks them non-temporal (each cached byte is read once).
template <bool NT>
__device__ __forceinline__ bf16x8 ld_kv(const uint16_t* ptr) {
  if constexpr (NT) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ptr)));
  } else {
    return ld_bf16x8(ptr);
  }
}

template <int D, bool NT>
__global__ __launch_bounds__(256, 2) void attn_split_kernel(AttnParams p) {
  constexpr int NC = D / 32;   // k-chunks of the QK product
  constexpr int NMT = D / 16;  // d-tiles of the PV product
  constexpr int LDO = D + 4;   // padded row of the LDS merge buffer

  __shared__ float sm_ml[kWaves][2][16];
  __shared__ __attribute__((aligned(16))) float sm_o[kWaves][16][LDO];

  const int bh = blockIdx.x;
  const int b = bh / p.Hkv;
  const int kvh = bh - b * p.Hkv;
  const int split = blockIdx.y;
  const int ctx = clamp_ctx(p, b);
  const int S = p.split_tokens;
  const int t0 = split * S;
  if (t0 > 0 && t0 >= ctx) return;  // split 0 always runs (it writes zeros when ctx == 0)
  const int t1 = min(t0 + S, ctx);
  const int nsplit = max(1, (ctx + S - 1) / S);
  const int jb0 = t0 / 16;
  const int nblk = (t1 - t0 + 15) / 16;
  const int npairs = (nblk + 1) / 2;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int r = lane & 15;   // MFMA row/col within the 16-wide tile
  const int qg = lane >> 4;  // lane group: which 8-wide k slice the lane feeds
  const int G = p.G;
  const int h0 = kvh * G;

  // Physical block ids of this split: lane i holds entry jb0 + i (split <= 64 blocks).
  int my_id = -1;
  if (lane < nblk) {
    my_id = p.bt[(size_t)b * p.max_blocks + jb0 + lane];
    if (my_id < 0 || my_id >= p.num_blocks) my_id = -1;
  }

  // q as the B operand of the QK product: column g = r, k = d in [c*32 + qg*8, +8).
  bf16x8 qf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    qf[c] = (r < G) ? ld_bf16x8(p.q + ((size_t)b * p.Hq + h0 + r) * D + c * 32 + qg * 8)
                    : zero_bf16x8();
  }

  // Token slots. QK tile row rr (lane rr loads it) holds token
  //   block (rr >> 3), offset ((rr >> 2) & 1) * 8 + (rr & 3)    [first product]
  //   ... + 4                                                  [second product]
  // so output rows 4*qg + i of the two products are tokens (qg&1)*8 + i and
  // (qg&1)*8 + 4 + i of block (qg >> 1): the 8 consecutive tokens whose V^T
  // slice this lane loads for the PV product.
  const int ksel = r >> 3;
  const int ktok = ((r >> 2) & 1) * 8 + (r & 3);
  const int vsel = qg >> 1;
  const int vtok = (qg & 1) * 8;

  float m_run = kNegInf;
  float l_run = 0.f;
  f32x4 acc[NMT];
#pragma unroll
  for (int mt = 0; mt < NMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int pr = wave; pr < npairs; pr += kWaves) {
    const int idA = __builtin_amdgcn_readlane(my_id, 2 * pr);
    const int idB = __builtin_amdgcn_readlane(my_id, 2 * pr + 1);
    const int tA = (jb0 + 2 * pr) * 16;

    bf16x8 k1[NC], k2[NC], vf[NMT];
    const int pk = ksel ? idB : idA;
    if (pk >= 0) {
      const uint16_t* kb = p.kc + ((size_t)pk * p.Hkv + kvh) * 16 * D + qg * 8;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        k1[c] = ld_kv<NT>(kb + ktok * D + c * 32);
        k2[c] = ld_kv<NT>(kb + (ktok + 4) * D + c * 32);
      }
    } else {
#pragma unroll
      for (int c = 0; c < NC; ++c) k1[c] = k2[c] = zero_bf16x8();
    }
    const int pv = vsel ? idB : idA;
    const int tb = tA + vsel * 16 + vtok;  // first token of this lane's 8-token slice
    const int nv = (pv >= 0) ? ctx - tb : 0;
    if (pv >= 0) {
      const uint16_t* vb = p.vc + ((size_t)pv * p.Hkv + kvh) * D * 16 + vtok;
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) vf[mt] = ld_kv<NT>(vb + (mt * 16 + r) * 16);
    } else {
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) vf[mt] = zero_bf16x8();
    }
    if (nv < 8) {  // tail of the last block (or a skipped block): zero V so 0 * NaN cannot leak
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) vf[mt] = keep_first(vf[mt], nv);
    }

    f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1[c], qf[c], s1, 0, 0, 0);
      s2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k2[c], qf[c], s2, 0, 0, 0);
    }

    float sv[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sv[i] = (i < nv) ? s1[i] * p.scale_log2 : kNegInf;
      sv[4 + i] = (4 + i < nv) ? s2[i] * p.scale_log2 : kNegInf;
    }
    float mx = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sv[i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    bf16x8 pb;
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const __bf16 e = static_cast<__bf16>(fast_exp2(sv[i] - m_use));
      pb[i] = e;
      ps += static_cast<float>(e);
    }
    l_run = l_run * alpha + ps;
    m_run = m_new;
#pragma unroll
    for (int mt = 0; mt < NMT; ++mt) {
      acc[mt] *= alpha;
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[mt], pb, acc[mt], 0, 0, 0);
    }
  }

  // Sum of the softmax denominators over the 4 lanes that share head g.
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  if (qg == 0) {
    sm_ml[wave][0][r] = m_run;
    sm_ml[wave][1][r] = l_run;
  }
#pragma unroll
  for (int mt = 0; mt < NMT; ++mt)
    *reinterpret_cast<f32x4*>(&sm_o[wave][r][mt * 16 + 4 * qg]) = acc[mt];
  __syncthreads();

  for (int it = tid; it < G * D; it += 256) {
    const int g = it / D;
    const int d = it - g * D;
    float M = sm_ml[0][0][g];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sm_ml[w][0][g]);
    const float Mu = (M == kNegInf) ? 0.f : M;
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float wt = fast_exp2(sm_ml[w][0][g] - Mu);
      L += wt * sm_ml[w][1][g];
      O += wt * sm_o[w][g][d];
    }
    const size_t row = (size_t)b * p.Hq + h0 + g;
    if (nsplit == 1) {
      p.out[row * D + d] = f2bf(L > 0.f ? O / L : 0.f);
    } else {
      const size_t prow = row * p.max_splits + split;
      p.part_o[prow * D + d] = O;
      if (d == 0) {
        p.part_ml[prow * 2 + 0] = M;
        p.part_ml[prow * 2 + 1] = L;
      }
    }
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One wave per (sequence, head). Lanes first reduce the split maxima and
// denominators in parallel, then each lane sums 4 consecutive d of every
// NG-th split (NG = 64 / (D/4) lane groups) with 16-byte loads, and the groups
// are combined with xor shuffles; the summation order is fixed.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  constexpr int D4 = D / 4;
  constexpr int NG = 64 / D4;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * kWaves + wave;  // (b, h)
  if (row >= p.B * p.Hq) return;
  const int b = row / p.Hq;
  const int ctx = clamp_ctx(p, b);
  const int nsplit = (ctx + p.split_tokens - 1) / p.split_tokens;
  if (nsplit <= 1) return;  // written by the split kernel
  const float* ml = p.part_ml + (size_t)row * p.max_splits * 2;
  float M = kNegInf;
  for (int s = lane; s < nsplit; s += 64) M = fmaxf(M, ml[2 * s]);
  M = wave_max(M);
  const float Mu = (M == kNegInf) ? 0.f : M;
  float L = 0.f;
  for (int s = lane; s < nsplit; s += 64) L += fast_exp2(ml[2 * s] - Mu) * ml[2 * s + 1];
  L = wave_sum(L);
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int grp = lane / D4, d4 = lane - grp * D4;
  const float* po = p.part_o + (size_t)row * p.max_splits * D + d4 * 4;
  f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int s = grp; s < nsplit; s += NG) O += fast_exp2(ml[2 * s] - Mu) * *reinterpret_cast<const f32x4*>(po + (size_t)s * D);
#pragma unroll
  for (int o = D4; o < 64; o <<= 1) {
#pragma unroll
    for (int e = 0; e < 4; ++e) O[e] += __shfl_xor(O[e], o);
  }
  if (grp == 0) {
    ushort4 v;
    v.x = f2bf(O[0] * inv);
    v.y = f2bf(O[1] * inv);
    v.z = f2bf(O[2] * inv);
    v.w = f2bf(O[3] * inv);
    *reinterpret_cast<ushort4*>(p.out + (size_t)row * D + d4 * 4) = v;
  }
}

int attn_split_tokens(const aflex_attn_args& a) {
  if (a.split_tokens > 0) return a.split_tokens;
  // Longer splits amortise each work-group's fixed cost (the block-id and q
  // loads ahead of its first K/V byte, the LDS merge, the partial write and
  // the merge kernel's share) but leave fewer work-groups to fill 256 CUs.
  // The context lengths stay on the device, so the work-group count is
  // bounded through max_context_len: the longest split whose bound still
  // leaves several rounds of work-groups.
  const long kv_rows = (long)a.B * a.Hkv;
  if (kv_rows * ((a.max_context_len + 1023) / 1024) >= 8192) return 1024;
  return kv_rows * ((a.max_context_len + 511) / 512) >= 4096 ? 512 : 256;
}

static int max_splits_of(const aflex_attn_args& a, int S) {
  return a.max_context_len > 0 ? (a.max_context_len + S - 1) / S : 1;
}

size_t attn_workspace_bytes(const aflex_attn_args& a) {
  const int S = attn_split_tokens(a);
  const size_t rows = (size_t)a.B * a.Hq * max_splits_of(a, S);
  if (max_splits_of(a, S) <= 1) return 256;
  return align_up(rows * a.D * sizeof(float), 256) + align_up(rows * 2 * sizeof(float), 256);
}

hipError_t launch_attn_decode(const aflex_attn_args& a, void* ws, hipStream_t stream, bool nt_kv) {
  AttnParams p;
  p.q = a.q;
  p.kc = a.k_cache;
  p.vc = a.v_cache;
  p.bt = a.block_table;
  p.cl = a.context_lens;
  p.out = a.out;
  p.B = a.B;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.G = a.Hq / a.Hkv;
  p.max_blocks = a.max_blocks_per_seq;
  p.num_blocks = a.num_blocks;
  p.max_ctx = a.max_context_len;
  p.split_tokens = attn_split_tokens(a);
  p.max_splits = max_splits_of(a, p.split_tokens);
  const float scale = a.scale != 0.f ? a.scale : 1.0f / sqrtf((float)a.D);
  p.scale_log2 = scale * kLog2e;
  const size_t rows = (size_t)a.B * a.Hq * p.max_splits;
  p.part_o = static_cast<float*>(ws);
  p.part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) +
                                       align_up(rows * a.D * sizeof(float), 256));
  dim3 grid(a.B * a.Hkv, p.max_splits);
  const unsigned merge_grid = (a.B * a.Hq + kWaves - 1) / kWaves;
  {
    ProfScope ps("attn_split", stream);
    if (a.D == 128) {
      if (nt_kv)
        attn_split_kernel<128, true><<<grid, 256, 0, stream>>>(p);
      else
        attn_split_kernel<128, false><<<grid, 256, 0, stream>>>(p);
    } else {
      if (nt_kv)
        attn_split_kernel<64, true><<<grid, 256, 0, stream>>>(p);
      else
        attn_split_kernel<64, false><<<grid, 256, 0, stream>>>(p);
    }
  }
  if (p.max_splits > 1) {
    ProfScope ps("attn_merge", stream);
    if (a.D == 128)
      attn_merge_kernel<128><<<merge_grid, 256, 0, stream>>>(p);
    else
      attn_merge_kernel<64><<<merge_grid, 256, 0, stream>>>(p);
  }
  return hipGetLastError();
}

}  // namespace aflex
