// MoE FFN block of a Mixtral layer, gfx950: RMSNorm, router GEMM, top-k MoE,
// optional residual.
//
// The FFN stage of the MoE model normalises the hidden state and computes the
// router logits before the experts run (Mixtral-8x7B, section 6.1). One
// work-group per token: it reads the row once, reduces the sum of squares,
// writes the normalised row in bf16 for the expert GEMMs and forms the E
// router logits from the fp32 normalised values (so routing decisions carry
// only fp32 summation error). All reductions are in a fixed order.
#include "common.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

constexpr int kNormMaxChunks = 8;  // 8 x 8 elements per thread: H <= 16384

__global__ __launch_bounds__(256) void rmsnorm_router_kernel(const uint16_t* __restrict__ x,
                                                             const uint16_t* __restrict__ gamma,
                                                             const uint16_t* __restrict__ wr, float eps, int H,
                                                             int E, uint16_t* __restrict__ xn,
                                                             float* __restrict__ logits,
                                                             float* __restrict__ logits_out) {
  __shared__ float red[4][kMaxRouterE + 1];
  const int t = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nch = H / 8;
  float v[kNormMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = tid + c * 256;
    if (ch < nch) {
      const uint4 u = *reinterpret_cast<const uint4*>(x + (size_t)t * H + ch * 8);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[c][e] = bf2f(static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16)));
        ss += v[c][e] * v[c][e];
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
  if (lane == 0) red[wave][0] = ss;
  __syncthreads();
  const float tot = (red[0][0] + red[1][0]) + (red[2][0] + red[3][0]);
  const float rstd = 1.f / sqrtf(tot / (float)H + eps);
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = tid + c * 256;
    if (ch < nch) {
      const uint4 g = *reinterpret_cast<const uint4*>(gamma + ch * 8);
      const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        v[c][e] = v[c][e] * rstd * bf2f(static_cast<uint16_t>(gw[e >> 1] >> ((e & 1) * 16)));
        const uint32_t b = f2bf(v[c][e]);
        if (e & 1)
          o[e >> 1] |= b << 16;
        else
          o[e >> 1] = b;
      }
      *reinterpret_cast<uint4*>(xn + (size_t)t * H + ch * 8) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
  for (int ex = 0; ex < E; ++ex) {
    float d = 0.f;
#pragma unroll
    for (int c = 0; c < kNormMaxChunks; ++c) {
      const int ch = tid + c * 256;
      if (ch < nch) {
        const uint4 wv = *reinterpret_cast<const uint4*>(wr + (size_t)ex * H + ch * 8);
        const uint32_t w[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) d += v[c][e] * bf2f(static_cast<uint16_t>(w[e >> 1] >> ((e & 1) * 16)));
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) d += __shfl_xor(d, o);
    if (lane == 0) red[wave][1 + ex] = d;
  }
  __syncthreads();
  if (tid < E) {
    const float l = (red[0][1 + tid] + red[1][1 + tid]) + (red[2][1 + tid] + red[3][1 + tid]);
    logits[(size_t)t * E + tid] = l;
    if (logits_out) logits_out[(size_t)t * E + tid] = l;
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
    rmsnorm_router_kernel<<<f.T, 256, 0, stream>>>(f.x, m.norm_weight, m.router_weight, m.eps, f.H, f.E, xn, logits,
                                                   m.router_logits_out);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  aflex_ffn_args g = f;
  g.x = xn;
  g.router_logits = logits;
  return launch_moe(g, moe_ws, stream, m.residual ? f.x : nullptr);
}

}  // namespace aflex
