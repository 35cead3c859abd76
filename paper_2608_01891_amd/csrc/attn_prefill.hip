// Causal prefill attention over packed prompts, gfx950.
//
// Prefill processes every prompt token at once and is dominated by dense
// contractions (section 2, "LLM Serving"; section 3.2 measures how its
// attention follows the GPU clock), so this kernel is built around the MFMA
// rate rather than HBM: for a 4096-token prompt each K/V row is reused by up
// to 4096 query rows.
//
// Work decomposition: one work-group per (query head, prompt, 128-row query
// tile); its 4 waves own 32 query rows each and walk the prompt's keys in
// tiles of 64 up to the causal limit of their rows. For batches with prompts
// of 2048 tokens or more and an even number of query heads per KV head, a
// work-group of 8 waves takes two heads of one KV group, so each staged K/V
// tile serves both (one such work-group per CU; shorter prompts run faster
// with two 4-wave work-groups per CU). Query tiles are dispatched
// longest-first (they are the slow index of the grid, reversed) so the short
// diagonal tiles fill the tail. When the number of head blocks is a multiple
// of 8 it is permuted so that the heads sharing one KV head run on the same
// XCD and share its L2.
//
// K and V tiles (64 keys x 128 d, row-major, 16-byte chunks XOR-swizzled by
// row so that both kinds of fragment read are free of bank conflicts) stream from HBM straight into double-buffered LDS (direct global->LDS
// loads); K runs one tile ahead of V. Per 64-key tile and wave, all products
// on v_mfma_f32_32x32x16_bf16:
//   S^T = K Q^T     two 32-key blocks x 8 k-steps of d; the query fragments
//                   (B operand) stay in registers for the whole kernel.
//   softmax         online, in the log2 domain: each lane holds 32 scores of
//                   one query row (an accumulator column), the other 32 sit in
//                   lane l ^ 32 (row maxima meet through v_permlane32_swap);
//                   O and l are rescaled only when a row's maximum rises more
//                   than 2^8 above the reference maximum. The row sum l adds
//                   the bf16-rounded weights that enter O (v_dot2 with (1, 1)),
//                   so numerator and denominator use the same weights.
//   O^T += V^T P^T  P^T is used straight from the S^T accumulator registers as
//                   the B operand (rounded to bf16); the V^T fragments (A
//                   operand) come from the row-major V tile through the
//                   transposing LDS read (ds_read_b64_tr_b16), in the key order
//                   the accumulator layout fixes.
// The scores of tile kt+1 are multiplied while the softmax of tile kt runs, so
// the MFMA and vector pipes of a wave overlap. The output tile is transposed
// back through LDS and written with 16-byte row-contiguous stores.
#include "common.h"
#include "gemm.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

namespace {

constexpr int kPM = 128;  // query rows per work-group
constexpr int kPN = 64;   // keys per tile
constexpr int kPD = 128;  // head dimension
constexpr int kTile = kPN * kPD * 2;  // bytes of one K or V tile
// Prompts at least this long run two query heads of a KV group per
// work-group (8 waves sharing each staged K/V tile, one work-group per CU);
// shorter ones one head (4 waves, two work-groups per CU).
constexpr int kTwoHeadMinLen = 2048;

struct PrefillParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* cu;
  uint16_t* out;
  int T, Hq, Hkv, G, ntiles;
  float c;  // softmax scale * log2(e)
};

typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Swizzle of the 16-byte chunks of a K or V tile row (256-byte rows, one
// 64-bank window each). Two reads must be conflict-free: 16-byte K fragments
// of 16 consecutive rows (any 16 distinct values do), and transposing reads in
// which each half-wave takes 64 contiguous bytes of 4 consecutive rows (the
// rows must land in different 64-byte quarters: bits 2-3 from row % 4).
__device__ __forceinline__ int kv_swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }
__device__ __forceinline__ uint32_t kv_off(int row, int chunk) { return row * 256 + ((chunk ^ kv_swz(row)) << 4); }

// Transposing LDS read: within each 16-lane group, lane i receives element
// i % 4 of the 4-element segment addressed by lane 4 j + i / 4, as element j.
__device__ __forceinline__ s16x4 lds_read_tr16(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((s16x4 __attribute__((address_space(3)))*)p);
}

// Maximum of a lane's value and lane l ^ 32's (one v_permlane32_swap).
__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

template <int HPW>
__global__ __launch_bounds__(256 * HPW, HPW == 1 ? 2 : 1) void attn_prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[4 * kTile];  // K0, K1, V0, V1

  const int nhb = p.Hq / HPW;
  int hb = blockIdx.x;
  if ((nhb & 7) == 0) hb = (hb & 7) * (nhb >> 3) + (hb >> 3);
  const int b = blockIdx.y;
  const int tile = p.ntiles - 1 - (int)blockIdx.z;
  int s1 = p.cu[b + 1], s0 = p.cu[b];
  s1 = min(max(s1, 0), p.T);
  s0 = min(max(s0, 0), s1);
  const int n = s1 - s0;
  const int q0 = tile * kPM;
  if (q0 >= n) return;

  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 31, hi = l >> 5;
  const int h = hb * HPW + (w >> 2);  // query head of this wave
  const int g = h / p.G;
  const int qr0 = q0 + (w & 3) * 32;  // first query row of this wave
  const int qi = qr0 + lr;         // this lane's query row (a column of S^T)
  const size_t qstride = (size_t)p.Hq * kPD, kvstride = (size_t)p.Hkv * kPD;

  // Query fragments: k-step ks holds d = 16 ks + 8 hi + [0, 8) of row qi.
  bf16x8 qf[kPD / 16];
  {
    const uint16_t* qrow = p.q + (size_t)(s0 + min(qi, n - 1)) * qstride + (size_t)h * kPD + hi * 8;
#pragma unroll
    for (int ks = 0; ks < kPD / 16; ++ks) qf[ks] = ld_bf16x8(qrow + ks * 16);
  }

  const int nkt = (min(n, q0 + kPM) + kPN - 1) / kPN;                // tiles the work-group stages
  const int wkt = qr0 < n ? min(nkt, min(qr0 + 31, n - 1) / kPN + 1) : 0;  // tiles this wave multiplies
  const uint16_t* kbase = p.k + (size_t)s0 * kvstride + (size_t)g * kPD;
  const uint16_t* vbase = p.v + (size_t)s0 * kvstride + (size_t)g * kPD;
  const uint32_t lds0 = lds_offset(smem);

  // Staging: wave-load i of thread tid fills slot i * 256 HPW + tid of the
  // tile, i.e. row i * 16 HPW + tid / 16 and stored chunk tid % 16; the logical
  // chunk is the same for all 4 / HPW wave-loads of a thread.
  const int srow = tid >> 4, schunk = (tid & 15) ^ kv_swz(srow);
  constexpr int RPL = 16 * HPW;  // tile rows per wave-load round of the work-group
  const size_t soff = (size_t)srow * kvstride + schunk * 8;
  auto issue = [&](const uint16_t* base, int kt, uint32_t lds) {
    lds += w * 1024;
    if (kt * kPN + kPN <= n) {
#pragma unroll
      for (int i = 0; i < 4 / HPW; ++i) lds_dma16(base + soff + (size_t)(kt * kPN + i * RPL) * kvstride, lds + i * 4096 * HPW);
    } else {  // tail tile: rows past the prompt re-read its last row (masked / weighted 0)
#pragma unroll
      for (int i = 0; i < 4 / HPW; ++i) {
        const int key = min(kt * kPN + i * RPL + srow, n - 1);
        lds_dma16(base + (size_t)key * kvstride + schunk * 8, lds + i * 4096 * HPW);
      }
    }
  };

  // Per-lane LDS byte offsets inside a tile. K fragment of k-step ks: row lr
  // (+32 for the second key block), chunk 2 ks + hi. Transposing V read of
  // d-block db: the lane addresses the 8-byte segment of row hi*4 + (l%16)/4
  // (+16 ks, +8 for the upper four keys) at d = 32 db + 16 ((l/16)%2) + 4 (l%4).
  // (Rows 32 and 16 further down share the swizzle, so those are immediates;
  // the upper four keys (+8 rows) do not, hence two transposing bases.)
  uint32_t k_off[kPD / 16], tr_lo[kPD / 32], tr_up[kPD / 32];
#pragma unroll
  for (int ks = 0; ks < kPD / 16; ++ks) k_off[ks] = kv_off(lr, ks * 2 + hi);
  {
    const int tr_row = hi * 4 + ((l & 15) >> 2);
#pragma unroll
    for (int db = 0; db < kPD / 32; ++db) {
      const int ch = db * 4 + ((l >> 4) & 1) * 2 + ((l & 3) >> 1);
      tr_lo[db] = kv_off(tr_row, ch) + (l & 1) * 8;
      tr_up[db] = kv_off(tr_row + 8, ch) + (l & 1) * 8;
    }
  }

  f32x16 oacc[kPD / 32];
#pragma unroll
  for (int db = 0; db < kPD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  float m_thr = kNegInf;  // m_run + 8 / c: a row maximum above it triggers a rescale
  const float thr_gap = 8.f / p.c;
  const bf16x2 ones2 = {(__bf16)1.f, (__bf16)1.f};
  f32x16 sc0, sc1, sn0, sn1;  // scores of the current tile and of the next one

#define AFLEX_QK(S0, S1, BUF)                                                                    \
  do {                                                                                           \
    _Pragma("unroll") for (int i = 0; i < 16; ++i) { S0[i] = 0.f; S1[i] = 0.f; }                 \
    const uint8_t* kl_ = smem + (BUF) * kTile;                                                   \
    _Pragma("unroll") for (int ks = 0; ks < kPD / 16; ++ks) {                                    \
      const bf16x8 a0_ = *reinterpret_cast<const bf16x8*>(kl_ + k_off[ks]);                      \
      const bf16x8 a1_ = *reinterpret_cast<const bf16x8*>(kl_ + k_off[ks] + 32 * 256);           \
      S0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0_, qf[ks], S0, 0, 0, 0);                    \
      S1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1_, qf[ks], S1, 0, 0, 0);                    \
    }                                                                                            \
  } while (0)

  // One key tile. KT is the tile, PAR = KT % 2 (a compile-time constant, so
  // every LDS address is a per-lane base plus an immediate), MASK whether any
  // key of the tile can lie past a row of the work-group or past the prompt.
  // SC0/SC1 hold the tile's scores on entry; SN0/SN1 receive the next tile's.
#define AFLEX_TILE(KT, PAR, MASK, SC0, SC1, SN0, SN1)                                         \
  do {                                                                                       \
    wait_vm0();                                                                              \
    __syncthreads();                                                                         \
    if ((KT) + 2 < nkt) issue(kbase, (KT) + 2, lds0 + (PAR) * kTile);                          \
    if ((KT) + 1 < nkt) issue(vbase, (KT) + 1, lds0 + (3 - (PAR)) * kTile);                    \
    if ((KT) < wkt) {                                                                        \
      if (MASK) {                                                                            \
        const int lim_ = min(qi, n - 1), kb0_ = (KT) * kPN;                                  \
        _Pragma("unroll") for (int i = 0; i < 16; ++i) {                                     \
          const int key_ = kb0_ + (i >> 2) * 8 + hi * 4 + (i & 3);                           \
          if (key_ > lim_) SC0[i] = kNegInf;                                                 \
          if (key_ + 32 > lim_) SC1[i] = kNegInf;                                            \
        }                                                                                    \
      }                                                                                      \
      float mx_ = fmaxf(SC0[0], SC1[0]);                                                     \
      _Pragma("unroll") for (int i = 1; i < 16; ++i) mx_ = fmaxf(fmaxf(mx_, SC0[i]), SC1[i]); \
      mx_ = max_across_halves(mx_);                                                          \
      if (__ballot(mx_ > m_thr) != 0) {                                                      \
        const float mnew_ = fmaxf(m_run, mx_);                                               \
        const float alpha_ = fast_exp2((m_run - mnew_) * p.c);                               \
        l_run *= alpha_;                                                                     \
        _Pragma("unroll") for (int db = 0; db < kPD / 32; ++db)                              \
            _Pragma("unroll") for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha_;            \
        m_run = mnew_;                                                                       \
        m_thr = m_run + thr_gap;                                                             \
      }                                                                                      \
      /* next tile's scores: independent of the exponentials below, which the */             \
      /* scheduler interleaves with them (dropped after a wave's last tile)   */             \
      AFLEX_QK(SN0, SN1, 1 - (PAR));                                                         \
      const float mc_ = m_run * p.c;                                                         \
      float lsum_ = 0.f;                                                                     \
      bf16x8 pb_[4];                                                                         \
      _Pragma("unroll") for (int ks = 0; ks < 4; ++ks) {                                     \
        f32x8 pv_;                                                                           \
        _Pragma("unroll") for (int e = 0; e < 8; ++e) {                                      \
          const float s_ = (ks < 2) ? SC0[(ks & 1) * 8 + e] : SC1[(ks & 1) * 8 + e];         \
          const float pe_ = fast_exp2(__builtin_fmaf(s_, p.c, -mc_));                        \
          pv_[e] = pe_;                                                                      \
        }                                                                                    \
        pb_[ks] = __builtin_convertvector(pv_, bf16x8);                                      \
        lsum_ = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb_[ks], pb_[ks], 0, 1), ones2, lsum_, false); \
        lsum_ = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb_[ks], pb_[ks], 2, 3), ones2, lsum_, false); \
        lsum_ = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb_[ks], pb_[ks], 4, 5), ones2, lsum_, false); \
        lsum_ = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb_[ks], pb_[ks], 6, 7), ones2, lsum_, false); \
      }                                                                                      \
      l_run += lsum_;                                                                        \
      /* O^T += V^T P^T: slot hi*8 + e of k-step ks is key ks*16 + (e/4)*8 + hi*4 + e%4 */    \
      const uint8_t* vl_ = smem + (2 + (PAR)) * kTile;                                       \
      _Pragma("unroll") for (int ks = 0; ks < 4; ++ks) {                                     \
        _Pragma("unroll") for (int db = 0; db < kPD / 32; ++db) {                            \
          const s16x4 lo_ = lds_read_tr16(vl_ + tr_lo[db] + ks * 4096);                      \
          const s16x4 up_ = lds_read_tr16(vl_ + tr_up[db] + ks * 4096);                      \
          const bf16x8 a_ = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo_, up_, 0, 1, 2, 3, 4, 5, 6, 7)); \
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_, pb_[ks], oacc[db], 0, 0, 0);  \
        }                                                                                    \
      }                                                                                      \
    }                                                                                        \
  } while (0)

  // Prologue: K(0), V(0), K(1) resident, S(0) computed.
  issue(kbase, 0, lds0);
  issue(vbase, 0, lds0 + 2 * kTile);
  if (nkt > 1) issue(kbase, 1, lds0 + kTile);
  wait_vm0();
  __syncthreads();
  if (wkt > 0) AFLEX_QK(sc0, sc1, 0);

  // Tiles below every row of the work-group and inside the prompt need no
  // mask; an even count keeps the two register sets and buffers in step.
  const int kfull = min(q0 / kPN, n / kPN) & ~1;
  int kt = 0;
  for (; kt < kfull; kt += 2) {
    AFLEX_TILE(kt, 0, false, sc0, sc1, sn0, sn1);
    AFLEX_TILE(kt + 1, 1, false, sn0, sn1, sc0, sc1);
  }
  for (; kt < nkt; kt += 2) {
    AFLEX_TILE(kt, 0, true, sc0, sc1, sn0, sn1);
    if (kt + 1 < nkt) AFLEX_TILE(kt + 1, 1, true, sn0, sn1, sc0, sc1);
  }
#undef AFLEX_TILE
#undef AFLEX_QK

  // Normalise and write: each wave transposes its 32 x 128 tile through its
  // own 8 KiB of LDS (chunk c of row r stored at chunk c ^ (r % 16)).
  const float lt = l_run + __shfl_xor(l_run, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  __syncthreads();
  uint8_t* osm = smem + w * 8192;
#pragma unroll
  for (int db = 0; db < kPD / 32; ++db)
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) {
      const int chunk = db * 4 + i4;
      const bf16x4 v4 = __builtin_convertvector(
          (f32x4){oacc[db][i4 * 4] * inv, oacc[db][i4 * 4 + 1] * inv, oacc[db][i4 * 4 + 2] * inv,
                  oacc[db][i4 * 4 + 3] * inv},
          bf16x4);
      *reinterpret_cast<bf16x4*>(osm + lr * 256 + ((chunk ^ (lr & 15)) << 4) + hi * 8) = v4;
    }
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int r = it * 4 + (l >> 4), c = l & 15;
    const int row = qr0 + r;
    const uint4 val = *reinterpret_cast<const uint4*>(osm + r * 256 + ((c ^ (r & 15)) << 4));
    if (row < n) *reinterpret_cast<uint4*>(p.out + (size_t)(s0 + row) * qstride + (size_t)h * kPD + c * 8) = val;
  }
}

}  // namespace

hipError_t launch_attn_prefill(const aflex_prefill_args& a, hipStream_t stream) {
  if (a.T == 0 || a.max_seqlen == 0) return hipSuccess;
  PrefillParams p;
  p.q = a.q;
  p.k = a.k;
  p.v = a.v;
  p.cu = a.cu_seqlens;
  p.out = a.out;
  p.T = a.T;
  p.Hq = a.Hq;
  p.Hkv = a.Hkv;
  p.G = a.Hq / a.Hkv;
  p.ntiles = (a.max_seqlen + kPM - 1) / kPM;
  const float scale = a.scale > 0.f ? a.scale : 1.f / sqrtf((float)a.D);
  p.c = scale * kLog2e;
  ProfScope ps("attn_prefill", stream);
  if (p.G % 2 == 0 && a.max_seqlen >= kTwoHeadMinLen)
    attn_prefill_kernel<2><<<dim3(a.Hq / 2, a.B, p.ntiles), 512, 0, stream>>>(p);
  else
    attn_prefill_kernel<1><<<dim3(a.Hq, a.B, p.ntiles), 256, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace aflex
