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
// tiles of 64 up to the causal limit of the tile. Query tiles are dispatched
// longest-first (they are the slow index of the grid, reversed) so the short
// diagonal tiles fill the tail. When Hq is a multiple of 8 the head index is
// permuted so that the heads sharing one KV head run on the same XCD and
// share its L2.
//
// Per 64-key tile and wave (v_mfma_f32_32x32x16_bf16 throughout):
//   S^T = K Q^T   two 32-key blocks x 8 k-steps of d; the query fragments
//                 (B operand) stay in registers for the whole kernel, K (A
//                 operand) is read from an LDS tile filled by direct
//                 global->LDS loads (double buffered, 16-byte chunks XOR
//                 swizzled by row so fragment reads are conflict-free).
//   softmax       online, in the log2 domain: each lane holds 32 scores of
//                 one query row (the accumulator's column), the other 32 sit
//                 in lane l ^ 32; O and l are rescaled only when a row's
//                 maximum rises more than 2^8 above the reference maximum.
//   O^T += V^T P^T  P^T is used straight from the S^T accumulator registers as
//                 the B operand (rounded to bf16), which fixes the order of the
//                 keys inside each 16-key k-step; V is transposed in registers
//                 (v_perm) while it is staged, into an LDS tile [d][key'] whose
//                 key order matches, so each A fragment is one 16-byte read.
// The output tile is transposed back through LDS and written with 16-byte
// row-contiguous stores.
#include "common.h"
#include "gemm.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

namespace {

constexpr int kPM = 128;  // query rows per work-group
constexpr int kPN = 64;   // keys per tile
constexpr int kPD = 128;  // head dimension

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

__device__ __forceinline__ void wait_vm8() { asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); }
__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Byte offset of 16-byte chunk `chunk` of row `row` in the K tile (256-byte
// rows, one 64-bank window each): 16 consecutive rows put a given chunk on 16
// distinct bank groups.
__device__ __forceinline__ uint32_t k_off(int row, int chunk) { return row * 256 + ((chunk ^ (row & 15)) << 4); }
// Byte offset of 16-byte chunk `chunk` of row d in the V^T tile (128-byte rows).
__device__ __forceinline__ uint32_t v_off(int d, int chunk) { return d * 128 + ((chunk ^ ((d + (d >> 3)) & 7)) << 4); }

__global__ __launch_bounds__(256, 2) void attn_prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * kPN * kPD * 2 + 2 * kPD * kPN * 2];
  uint8_t* const ksm = smem;                         // 2 x 16 KiB K tiles [key][d]
  uint8_t* const vsm = smem + 2 * kPN * kPD * 2;     // 2 x 16 KiB V^T tiles [d][key']

  int h = blockIdx.x;
  if ((p.Hq & 7) == 0) h = (h & 7) * (p.Hq >> 3) + (h >> 3);
  const int b = blockIdx.y;
  const int tile = p.ntiles - 1 - (int)blockIdx.z;
  int s1 = p.cu[b + 1], s0 = p.cu[b];
  s1 = min(max(s1, 0), p.T);
  s0 = min(max(s0, 0), s1);
  const int n = s1 - s0;
  const int q0 = tile * kPM;
  if (q0 >= n) return;

  const int g = h / p.G;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 31, hi = l >> 5;
  const int qr0 = q0 + w * 32;     // first query row of this wave
  const int qi = qr0 + lr;         // this lane's query row (a column of S^T)
  const size_t qstride = (size_t)p.Hq * kPD, kvstride = (size_t)p.Hkv * kPD;

  // Query fragments: k-step ks holds d = 16 ks + 8 hi + [0, 8) of row qi.
  bf16x8 qf[kPD / 16];
  {
    const uint16_t* qrow = p.q + (size_t)(s0 + min(qi, n - 1)) * qstride + (size_t)h * kPD + hi * 8;
#pragma unroll
    for (int ks = 0; ks < kPD / 16; ++ks) qf[ks] = ld_bf16x8(qrow + ks * 16);
  }

  const int kend = min(n, q0 + kPM);
  const int nkt = (kend + kPN - 1) / kPN;
  const uint16_t* kbase = p.k + (size_t)s0 * kvstride + (size_t)g * kPD;
  const uint16_t* vbase = p.v + (size_t)s0 * kvstride + (size_t)g * kPD;
  const uint32_t ksm_lds = lds_offset(ksm);

  // K staging: wave-load i of thread tid fills slot i * 256 + tid, i.e. row
  // i * 16 + tid / 16 and stored chunk tid % 16 of the tile; the logical chunk
  // is the same for all four wave-loads of a thread.
  const int krow = tid >> 4, kchunk = (tid & 15) ^ krow;
  const uint16_t* kp = kbase + (size_t)krow * kvstride + kchunk * 8;
  auto issue_k = [&](int kt, int buf) {
    const uint32_t lds = ksm_lds + buf * 16384 + w * 1024;
    if (kt * kPN + kPN <= n) {
#pragma unroll
      for (int i = 0; i < 4; ++i) lds_dma16(kp + (size_t)(kt * kPN + i * 16) * kvstride, lds + i * 4096);
    } else {  // tail tile: rows past the prompt re-read its last row (their scores are masked)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = min(kt * kPN + i * 16 + krow, n - 1);
        lds_dma16(kbase + (size_t)key * kvstride + kchunk * 8, lds + i * 4096);
      }
    }
  };
  // V staging: thread tid loads keys 4a .. 4a+3 (a = tid / 16) at d = 8 (tid % 16) + [0, 8).
  const int va = tid >> 4, vdc = tid & 15;
  const uint16_t* vp = vbase + (size_t)(va * 4) * kvstride + vdc * 8;
  uint4 vr[4];
  auto load_v = [&](int kt) {
    if (kt * kPN + kPN <= n) {
#pragma unroll
      for (int j = 0; j < 4; ++j) vr[j] = *reinterpret_cast<const uint4*>(vp + (size_t)(kt * kPN + j) * kvstride);
    } else {  // tail tile: rows past the prompt re-read its last row (their weights are 0)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = min(kt * kPN + va * 4 + j, n - 1);
        vr[j] = *reinterpret_cast<const uint4*>(vbase + (size_t)key * kvstride + vdc * 8);
      }
    }
  };
  // Keys 4a' .. 4a'+3 of a 16-key group sit at positions (a' % 2) * 8 + (a' / 2) * 4 + [0, 4)
  // of that group in the V^T tile: the order in which the S^T accumulator holds them.
  auto store_vt = [&](int buf) {
    const int grp = va >> 2, ap = va & 3;
    const int chunk = grp * 2 + (ap & 1), within = (ap >> 1) * 8;
    const uint32_t w0[4] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w};
    const uint32_t w1[4] = {vr[1].x, vr[1].y, vr[1].z, vr[1].w};
    const uint32_t w2[4] = {vr[2].x, vr[2].y, vr[2].z, vr[2].w};
    const uint32_t w3[4] = {vr[3].x, vr[3].y, vr[3].z, vr[3].w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
      uint2 val;
      val.x = __builtin_amdgcn_perm(w1[e >> 1], w0[e >> 1], sel);
      val.y = __builtin_amdgcn_perm(w3[e >> 1], w2[e >> 1], sel);
      const int d = vdc * 8 + e;
      *reinterpret_cast<uint2*>(vsm + buf * 16384 + v_off(d, chunk) + within) = val;
    }
  };

  f32x16 oacc[kPD / 32];
#pragma unroll
  for (int db = 0; db < kPD / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;
  float m_run = kNegInf, l_run = 0.f;

  issue_k(0, 0);
  load_v(0);
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt > 0) __syncthreads();  // every wave is done with tile kt - 1
    store_vt(buf);
    if (kt + 1 < nkt) {
      issue_k(kt + 1, buf ^ 1);
      load_v(kt + 1);
      wait_vm8();  // this thread's part of K tile kt has landed
    } else {
      wait_vm0();
    }
    __syncthreads();

    const int kb0 = kt * kPN;
    if (kb0 > qr0 + 31 || qr0 >= n) continue;  // every key of the tile is masked for this wave

    // S^T = K Q^T
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[kb][i] = 0.f;
    const uint8_t* kt_lds = ksm + buf * 16384;
#pragma unroll
    for (int ks = 0; ks < kPD / 16; ++ks) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kt_lds + k_off(kb * 32 + lr, ks * 2 + hi));
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], sacc[kb], 0, 0, 0);
      }
    }

    // Mask keys past the query row or past the prompt (diagonal and tail tiles only).
    if (kb0 + kPN - 1 > qr0 || kb0 + kPN > n) {
      const int lim = min(qi, n - 1);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kb0 + kb * 32 + (i >> 2) * 8 + hi * 4 + (i & 3);
          if (key > lim) sacc[kb][i] = kNegInf;
        }
    }

    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // The reference maximum m_run only moves when a row's scores exceed it by
    // more than 2^8 in the exponent: O and l share the reference, so the
    // normalised result does not depend on it, and the weights stay <= 256.
    if (__ballot((mx - m_run) * p.c > 8.f) != 0) {
      const float mnew = fmaxf(m_run, mx);
      const float alpha = fast_exp2((m_run - mnew) * p.c);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < kPD / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
      m_run = mnew;
    }
    const float mc = m_run * p.c;
    float lsum = 0.f;
    bf16x8 pb[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      f32x8 pv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float pe = fast_exp2(__builtin_fmaf(sacc[ks >> 1][(ks & 1) * 8 + e], p.c, -mc));
        lsum += pe;
        pv[e] = pe;
      }
      pb[ks] = __builtin_convertvector(pv, bf16x8);
    }
    l_run += lsum;

    // O^T += V^T P^T
    const uint8_t* vt_lds = vsm + buf * 16384;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int db = 0; db < kPD / 32; ++db) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(vt_lds + v_off(db * 32 + lr, ks * 2 + hi));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
      }
    }
  }

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
  attn_prefill_kernel<<<dim3(a.Hq, a.B, p.ntiles), 256, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace aflex
