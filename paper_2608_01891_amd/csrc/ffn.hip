// Dense SwiGLU FFN, gfx950: y = (SiLU(x W_g^T) * (x W_u^T)) W_d^T.
//
// The FFN of the dense model the paper evaluates (Qwen3-32B, section 6.1);
// its decode-batch behaviour -- weight-streaming at small batch, MFMA-bound at
// large batch -- is the FFN sensitivity the paper characterises (section 1,
// section 3.2).
//
// Steps:
//   1. gate/up GEMM with the fused SwiGLU epilogue -> h [T, I] bf16 (workspace)
//   2. down GEMM -> fp32 split-K partials (or bf16 y directly when one split)
//   3. fixed-order sum of the partials -> y [T, H] bf16
#include "ffn_plan.h"
#include "gemm.h"
#include "kernels.h"
#include "profile.h"

namespace aflex {

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ P, long long split_stride,
                                                            int splits, long long n4,
                                                            uint16_t* __restrict__ y,
                                                            const uint16_t* __restrict__ residual) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  // Four slices are loaded before any is added (indices past the last slice
  // re-read it and are not added), so a call with many splits waits for one
  // memory round trip per four slices, not per slice. The sum keeps slice
  // order and starts from -0, which leaves the first slice's value unchanged.
  constexpr int kBatch = 4;
  f32x4 s = {-0.f, -0.f, -0.f, -0.f};
  for (int k0 = 0; k0 < splits; k0 += kBatch) {
    f32x4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      v[u] = *reinterpret_cast<const f32x4*>(P + min(k0 + u, splits - 1) * split_stride + i * 4);
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (k0 + u < splits) s += v[u];
  }
  if (residual) {  // added after the split sum, before the one rounding
    const ushort4 r = *reinterpret_cast<const ushort4*>(residual + i * 4);
    s[0] += bf2f(r.x);
    s[1] += bf2f(r.y);
    s[2] += bf2f(r.z);
    s[3] += bf2f(r.w);
  }
  ushort4 o;
  o.x = f2bf(s[0]);
  o.y = f2bf(s[1]);
  o.z = f2bf(s[2]);
  o.w = f2bf(s[3]);
  *reinterpret_cast<ushort4*>(y + i * 4) = o;
}

size_t swiglu_workspace_bytes(const aflex_ffn_args& f) {
  const FfnPlan pl = plan_dense(f.T, f.H, f.I);
  size_t b = align_up((size_t)f.T * f.I * 2, 256);
  if (pl.down_splits > 1) b += align_up((size_t)pl.down_splits * f.T * f.H * 4, 256);
  return b;
}

hipError_t launch_swiglu(const aflex_ffn_args& f, void* ws, hipStream_t stream) {
  const FfnPlan pl = plan_dense(f.T, f.H, f.I);
  uint16_t* h = static_cast<uint16_t*>(ws);
  float* P = reinterpret_cast<float*>(static_cast<char*>(ws) + align_up((size_t)f.T * f.I * 2, 256));

  GemmParams g = {};
  g.A = f.x;
  g.lda = f.H;
  g.B0 = f.w_gate;
  g.B1 = f.w_up;
  g.ldb = f.H;
  g.N = f.I;
  g.K = f.H;
  g.k_per_split = f.H;
  g.splits = 1;
  g.M = f.T;
  g.max_mtiles = (f.T + pl.bm - 1) / pl.bm;
  g.n_ntiles = (f.I + gate_bn(pl.bm) - 1) / gate_bn(pl.bm);
  g.mt_major = 0;
  g.C = h;
  g.ldc = f.I;
  const bool once = f.T <= pl.bm;
  hipError_t e = launch_gate_up(pl.bm, once, g, stream);
  if (e != hipSuccess) return e;

  GemmParams d = {};
  d.A = h;
  d.lda = f.I;
  d.B0 = f.w_down;
  d.ldb = f.I;
  d.N = f.H;
  d.K = f.I;
  d.k_per_split = pl.down_kps;
  d.splits = pl.down_splits;
  d.M = f.T;
  d.max_mtiles = (f.T + pl.bm - 1) / pl.bm;
  d.n_ntiles = (f.H + down_bn(pl.bm) - 1) / down_bn(pl.bm);
  d.mt_major = 0;
  d.C = f.y;
  d.ldc = f.H;
  d.P = P;
  d.p_split_stride = (long long)f.T * f.H;
  d.ldp = f.H;
  e = launch_down(pl.bm, pl.down_splits > 1, once, d, stream);
  if (e != hipSuccess || pl.down_splits == 1) return e;
  const long long n4 = (long long)f.T * f.H / 4;
  ProfScope ps("splitk_reduce", stream);
  splitk_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, stream>>>(P, d.p_split_stride, pl.down_splits, n4,
                                                                       f.y, nullptr);
  return hipGetLastError();
}

// Linear layer y = x W^T (+ residual): the down-GEMM tiles with split-K and
// the same fixed-order reduction (bf16 out directly when a single split
// suffices); the optional residual is added before the one rounding.
size_t linear_workspace_bytes(const aflex_linear_args& l) {
  const FfnPlan pl = plan_dense(l.T, l.N, l.K);
  return pl.down_splits > 1 ? align_up((size_t)pl.down_splits * l.T * l.N * 4, 256) : 256;
}

hipError_t launch_linear(const aflex_linear_args& l, void* ws, hipStream_t stream, const uint16_t* residual) {
  const FfnPlan pl = plan_dense(l.T, l.N, l.K);
  float* P = static_cast<float*>(ws);
  GemmParams d = {};
  d.A = l.x;
  d.lda = l.K;
  d.B0 = l.w;
  d.ldb = l.K;
  d.N = l.N;
  d.K = l.K;
  d.k_per_split = pl.down_kps;
  d.splits = pl.down_splits;
  d.M = l.T;
  d.max_mtiles = (l.T + pl.bm - 1) / pl.bm;
  d.n_ntiles = (l.N + down_bn(pl.bm) - 1) / down_bn(pl.bm);
  d.mt_major = 0;
  d.C = l.y;
  d.ldc = l.N;
  d.P = P;
  d.p_split_stride = (long long)l.T * l.N;
  d.ldp = l.N;
  d.R = residual;
  hipError_t e = launch_down(pl.bm, pl.down_splits > 1, l.T <= pl.bm, d, stream);
  if (e != hipSuccess || pl.down_splits == 1) return e;
  const long long n4 = (long long)l.T * l.N / 4;
  ProfScope ps("splitk_reduce", stream);
  splitk_reduce_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, stream>>>(P, d.p_split_stride, pl.down_splits, n4,
                                                                       l.y, residual);
  return hipGetLastError();
}

}  // namespace aflex
