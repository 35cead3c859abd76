// bf16 MFMA GEMM C = A . B^T for the FFN contractions, gfx950.
//
// A [rows, K] holds tokens (optionally gathered through an index list, which
// is how the MoE reads its token-permuted input without materialising it),
// B [N, K] holds weights in the [out_features, in_features] layout, so both
// operands have the contraction index contiguous and every MFMA operand is
// one 16-byte LDS read. Tiles of BM x BN x 64 are staged global -> registers
// -> LDS with a double buffer (the next k-step's loads are in flight while
// the current one is multiplied) using v_mfma_f32_16x16x32_bf16.
//
// Variants (template flags):
//   DUAL    two weight matrices (gate, up) share the A tile; the epilogue
//           applies SiLU(gate) * up and stores bf16 (the fused SwiGLU step).
//   OUT_F32 store the fp32 accumulator into split-K partials (one slice per
//           split; a later kernel sums the slices in a fixed order).
//   neither store bf16.
//
// Work decomposition: a 1-D grid over (m-tile, n-tile, k-split). Work-groups
// are dispatched round-robin over the 8 XCDs; the logical tile index is
// remapped so that consecutive tiles (which share an A tile, or for dense
// GEMMs a weight tile across m-tiles) land on the same XCD and its L2.
// m-tiles come either from a dense row count or from a device-side tile map
// of (expert, first row, end row) triples written by the MoE routing kernel;
// work-groups beyond the map's device-side count exit at once, so the grid is
// sized for the worst case without a host synchronisation.
#pragma once
#include "common.h"

namespace aflex {

struct GemmParams {
  const uint16_t* A;
  int lda;
  const int32_t* gather;  // optional: logical row r reads A row gather[r] / gather_div
  int gather_div;
  const uint16_t* B0;
  const uint16_t* B1;     // second weight matrix (DUAL only)
  int ldb;
  long long b_expert_stride;  // elements between experts' weight matrices
  int N, K;
  int k_per_split, splits;
  int M;                      // dense row count (tile_map == nullptr)
  const int32_t* tile_map;    // [max_mtiles][3] = (expert, row_begin, row_end)
  const int32_t* num_mtiles;  // device count of valid tile_map entries
  int max_mtiles;
  int n_ntiles;
  int mt_major;               // 1: m-tile is the slow index of the tile order
  uint16_t* C;                // bf16 output [rows, ldc]
  int ldc;
  float* P;                   // fp32 split-K partials [splits][rows][ldp]
  long long p_split_stride;
  int ldp;
};

__device__ __forceinline__ int xcd_remap(int w, int nwg) {
  const int q = nwg >> 3, rem = nwg & 7, x = w & 7, j = w >> 3;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + j;
}

template <int BM, int BN, int WM, int WN, bool DUAL, bool OUT_F32>
__global__ __launch_bounds__(256, 2) void gemm_nt_kernel(GemmParams p) {
  constexpr int BK = 64;
  constexpr int LDK = BK + 8;  // padded LDS row (144 B): conflict-free 16-byte fragment reads
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int A_CH = BM * 8 / 256;
  constexpr int B_CH = BN * 8 / 256;
  static_assert(WM * WN == 4, "4 waves per work-group");
  static_assert(TM >= 1 && TN >= 1 && A_CH >= 1 && B_CH >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) uint16_t smA[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t smB[2][NB][BN * LDK];

  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int split = t % p.splits;
  const int rest = t / p.splits;
  int mt, nt;
  if (p.mt_major) {
    nt = rest % p.n_ntiles;
    mt = rest / p.n_ntiles;
  } else {
    mt = rest % p.max_mtiles;
    nt = rest / p.max_mtiles;
  }
  int expert = 0, row0, row1;
  if (p.tile_map) {
    if (mt >= *p.num_mtiles) return;
    expert = p.tile_map[3 * mt + 0];
    row0 = p.tile_map[3 * mt + 1];
    row1 = p.tile_map[3 * mt + 2];
  } else {
    row0 = mt * BM;
    row1 = min(row0 + BM, p.M);
  }
  const int n0 = nt * BN;
  const int kb = split * p.k_per_split;
  const int ke = min(p.K, kb + p.k_per_split);
  const int nk = (ke - kb) / BK;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r = lane & 15, qg = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;

  // Per-thread global source rows (fixed over k).
  const uint16_t* a_src[A_CH];
#pragma unroll
  for (int i = 0; i < A_CH; ++i) {
    const int c = tid + i * 256;
    const int row = row0 + (c >> 3);
    const int col = (c & 7) * 8;
    if (row < row1) {
      const int src = p.gather ? p.gather[row] / p.gather_div : row;
      a_src[i] = p.A + (size_t)src * p.lda + kb + col;
    } else {
      a_src[i] = nullptr;
    }
  }
  const uint16_t* b_src[NB][B_CH];
#pragma unroll
  for (int i = 0; i < B_CH; ++i) {
    const int c = tid + i * 256;
    const int n = n0 + (c >> 3);
    const int col = (c & 7) * 8;
    const size_t off = (size_t)expert * p.b_expert_stride + (size_t)n * p.ldb + kb + col;
    b_src[0][i] = (n < p.N) ? p.B0 + off : nullptr;
    if (DUAL) b_src[NB - 1][i] = (n < p.N) ? p.B1 + off : nullptr;
  }

  uint4 ra[A_CH], rb[NB][B_CH];
  auto load_global = [&](int kt) {
    const int ko = kt * BK;
#pragma unroll
    for (int i = 0; i < A_CH; ++i)
      ra[i] = a_src[i] ? *reinterpret_cast<const uint4*>(a_src[i] + ko) : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < B_CH; ++i)
        rb[nb][i] = b_src[nb][i] ? *reinterpret_cast<const uint4*>(b_src[nb][i] + ko)
                                 : make_uint4(0, 0, 0, 0);
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<uint4*>(&smA[buf][(c >> 3) * LDK + (c & 7) * 8]) = ra[i];
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < B_CH; ++i) {
        const int c = tid + i * 256;
        *reinterpret_cast<uint4*>(&smB[buf][nb][(c >> 3) * LDK + (c & 7) * 8]) = rb[nb][i];
      }
  };

  f32x4 acc[NB][TM][TN];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[nb][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    load_global(0);
    store_lds(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      bf16x8 af[TM], bfr[NB][TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(
            &smA[buf][(wm * WTM + i * 16 + r) * LDK + kk * 32 + qg * 8]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[nb][j] = *reinterpret_cast<const bf16x8*>(
              &smB[buf][nb][(wn * WTN + j * 16 + r) * LDK + kk * 32 + qg * 8]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[nb][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[nb][j], acc[nb][i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds rows (4*qg + e) and column r of every 16x16 tile.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * WTN + j * 16 + r;
      if (col >= p.N) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0 + wm * WTM + i * 16 + 4 * qg + e;
        if (row >= row1) continue;
        if (OUT_F32) {
          p.P[(size_t)split * p.p_split_stride + (size_t)row * p.ldp + col] = acc[0][i][j][e];
        } else if (DUAL) {
          const float g = acc[0][i][j][e];
          const float u = acc[NB - 1][i][j][e];
          const float h = g / (1.f + __expf(-g)) * u;
          p.C[(size_t)row * p.ldc + col] = f2bf(h);
        } else {
          p.C[(size_t)row * p.ldc + col] = f2bf(acc[0][i][j][e]);
        }
      }
    }
  }
}

}  // namespace aflex
