// MoE FFN block of a Mixtral layer, gfx950: RMSNorm, router GEMM, top-k MoE,
// optional residual.
//
// The FFN stage of the MoE model normalises the hidden state and computes the
// router logits before the experts run (Mixtral-8x7B, section 6.1). One
// work-group per token reads the row, its RMSNorm gain and the router rows in
// one batch of loads: the router logits are formed as
//   logits[e] = rstd * sum_h (x_h * gamma_h) * W_r[e, h],
// the same value as the dot product of the normalised row with W_r[e] (so
// routing decisions carry only fp32 summation error), which lets the sums of
// squares and of the E router products be reduced together instead of each
// router product waiting for the normalisation. The normalised row is then
// written in bf16 for the expert GEMMs. All reductions run in a fixed order.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

// MAXC chunks of 8 elements per thread: H <= MAXC * 2048.
template <int MAXC>
__global__ __launch_bounds__(256) void rmsnorm_router_kernel(const uint16_t* __restrict__ x,
                                                             const uint16_t* __restrict__ gamma,
                                                             const uint16_t* __restrict__ wr, float eps, int H,
                                                             int E, uint16_t* __restrict__ xn,
                                                             float* __restrict__ logits,
                                                             float* __restrict__ logits_out) {
  constexpr int EG = MAXC <= 2 ? 8 : 16 / MAXC;  // router rows per group of loads
  __shared__ float red[4][kMaxRouterE + 1];
  const int t = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nch = H / 8;
  float v[MAXC][8], xg[MAXC][8];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int ch = tid + c * 256;
    if (ch < nch) {
      const uint4 u = *reinterpret_cast<const uint4*>(x + (size_t)t * H + ch * 8);
      const uint4 gq = *reinterpret_cast<const uint4*>(gamma + ch * 8);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
      const uint32_t gw[4] = {gq.x, gq.y, gq.z, gq.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[c][e] = bf2f(static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16)));
        xg[c][e] = v[c][e] * bf2f(static_cast<uint16_t>(gw[e >> 1] >> ((e & 1) * 16)));
        ss += v[c][e] * v[c][e];
      }
    }
  }
  for (int e0 = 0; e0 < E; e0 += EG) {
    float d[EG];
#pragma unroll
    for (int j = 0; j < EG; ++j) {
      d[j] = 0.f;
      if (e0 + j < E) {
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
          const int ch = tid + c * 256;
          if (ch < nch) {
            const uint4 wv = *reinterpret_cast<const uint4*>(wr + (size_t)(e0 + j) * H + ch * 8);
            const uint32_t w[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) d[j] += xg[c][e] * bf2f(static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16)));
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < EG; ++j) {
      float r = d[j];
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) r += __shfl_xor(r, o);
      if (lane == 0 && e0 + j < E) red[wave][1 + e0 + j] = r;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if (lane == 0) red[wave][0] = ss;
  __syncthreads();
  const float tot = (red[0][0] + red[1][0]) + (red[2][0] + red[3][0]);
  const float rstd = 1.f / sqrtf(tot / (float)H + eps);
  if (tid < E) {
    const float l = rstd * ((red[0][1 + tid] + red[1][1 + tid]) + (red[2][1 + tid] + red[3][1 + tid]));
    logits[(size_t)t * E + tid] = l;
    if (logits_out) logits_out[(size_t)t * E + tid] = l;
  }
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int ch = tid + c * 256;
    if (ch < nch) {
      const uint4 gq = *reinterpret_cast<const uint4*>(gamma + ch * 8);
      const uint32_t gw[4] = {gq.x, gq.y, gq.z, gq.w};
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float y = v[c][e] * rstd * bf2f(static_cast<uint16_t>(gw[e >> 1] >> ((e & 1) * 16)));
        const uint32_t b = f2bf(y);
        if (e & 1)
          o[e >> 1] |= b << 16;
        else
          o[e >> 1] = b;
      }
      *reinterpret_cast<uint4*>(xn + (size_t)t * H + ch * 8) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

size_t moe_block_workspace_bytes(const aflex_moe_block_args& m) {
  const aflex_ffn_args& f = m.ffn;
  return align_up((size_t)f.T * f.H * 2, 256) + align_up((size_t)f.T * f.E * 4, 256) + moe_workspace_bytes(f);
}

hipError_t launch_moe_block(const aflex_moe_block_args& m, void* ws, hipStream_t stream) {
  const aflex_ffn_args& f = m.ffn;
  char* w = static_cast<char*>(ws);
  uint16_t* xn = reinterpret_cast<uint16_t*>(w);
  float* logits = reinterpret_cast<float*>(w + align_up((size_t)f.T * f.H * 2, 256));
  void* moe_ws = w + align_up((size_t)f.T * f.H * 2, 256) + align_up((size_t)f.T * f.E * 4, 256);
  {
    ProfScope ps("rmsnorm_router", stream);
    if (f.H <= 2048)
      rmsnorm_router_kernel<1><<<f.T, 256, 0, stream>>>(f.x, m.norm_weight, m.router_weight, m.eps, f.H, f.E, xn,
                                                        logits, m.router_logits_out);
    else if (f.H <= 4096)
      rmsnorm_router_kernel<2><<<f.T, 256, 0, stream>>>(f.x, m.norm_weight, m.router_weight, m.eps, f.H, f.E, xn,
                                                        logits, m.router_logits_out);
    else if (f.H <= 8192)
      rmsnorm_router_kernel<4><<<f.T, 256, 0, stream>>>(f.x, m.norm_weight, m.router_weight, m.eps, f.H, f.E, xn,
                                                        logits, m.router_logits_out);
    else
      rmsnorm_router_kernel<8><<<f.T, 256, 0, stream>>>(f.x, m.norm_weight, m.router_weight, m.eps, f.H, f.E, xn,
                                                        logits, m.router_logits_out);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  aflex_ffn_args g = f;
  g.x = xn;
  g.router_logits = logits;
  return launch_moe(g, moe_ws, stream, m.residual ? f.x : nullptr);
}

}  // namespace aflex
