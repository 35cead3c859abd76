// bf16 MFMA GEMM C = A . B^T for the FFN contractions, gfx950.
//
// A [rows, K] holds tokens (optionally gathered through an index list, which
// is how the MoE reads its token-permuted input without materialising it),
// B [N, K] holds weights in the [out_features, in_features] layout, so both
// operands have the contraction index contiguous and every MFMA operand is
// one 16-byte LDS read. Tiles of BM x BN x 64 stream from HBM straight into a
// ring of 3-4 LDS stages (global_load_lds_dwordx4, no register staging), so
// the loads of the next k-steps are in flight while kt is multiplied
// (v_mfma_f32_16x16x32_bf16). At decode batch sizes these GEMMs stream
// weights, so the depth of the load pipeline, not the MFMA rate, sets their
// speed.
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

// 32-bit LDS offset of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<size_t>((__attribute__((address_space(3))) const void*)p));
}

// Direct HBM -> LDS load of 16 bytes per lane: lane l writes LDS bytes
// [lds + 16 l, lds + 16 l + 16). Issued as inline assembly so the compiler's
// wait-count pass does not serialise it against reads of other LDS stages;
// callers order it with explicit s_waitcnt vmcnt and barriers.
__device__ __forceinline__ void lds_dma16(const void* gptr, uint32_t lds) {
  const uint32_t lds_s = __builtin_amdgcn_readfirstlane(lds);  // uniform across the wave
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(lds_s) : "memory", "m0");
}

__device__ __forceinline__ int xcd_remap(int w, int nwg) {
  const int q = nwg >> 3, rem = nwg & 7, x = w & 7, j = w >> 3;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + j;
}

template <int BM, int BN, int WM, int WN, bool DUAL, bool OUT_F32>
__global__ __launch_bounds__(256, BM >= 128 ? 1 : 2) void gemm_nt_kernel(GemmParams p) {
  constexpr int BK = 64;  // one LDS row = 64 bf16 = 128 B = 8 chunks of 16 B
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int ROWS = BM + NB * BN;   // LDS rows per stage: A tile, then the B tile(s)
  constexpr int INS = ROWS / 8;        // 1 KiB wave-loads per stage (8 rows each)
  constexpr int IPW = INS / 4;         // per wave
  constexpr int STAGE_BYTES = ROWS * BK * 2;
  // As many stages as fit in 80 KiB (two work-groups per CU share its 160 KiB),
  // at least three; BM >= 128 runs one work-group per CU with four stages.
  constexpr int STAGES = BM >= 128 ? 4 : (81920 / STAGE_BYTES < 3 ? 3 : 81920 / STAGE_BYTES);
  static_assert(WM * WN == 4, "4 waves per work-group");
  static_assert(TM >= 1 && TN >= 1 && INS % 4 == 0, "tile shape");
  static_assert((STAGES - 2) * IPW < 64, "vmcnt range");

  // Ring of STAGES buffers filled by direct global->LDS loads: lane l of a
  // wave-load writes the 16 bytes at slot base + l. Slot s of a stage holds
  // row s >> 3, 16-byte chunk (s & 7) ^ ((row >> 1) & 7) of the tile, so the 16
  // rows of an MFMA fragment read fall on distinct bank groups.
  __shared__ __attribute__((aligned(16))) uint16_t sm[STAGES][ROWS * BK];

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

  // Global source of each of this lane's wave-loads (fixed over k). Rows past
  // the tile (A rows >= row1, weight rows >= N) read a valid row instead; their
  // products land in output rows/columns that are never stored.
  const uint16_t* src[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int slot = (wave + 4 * j) * 64 + lane;
    const int row = slot >> 3;
    const int ch = (slot & 7) ^ ((row >> 1) & 7);
    const uint16_t* base;
    if (row < BM) {
      const int g = (row0 + row < row1) ? row0 + row : row0;
      const int srow = p.gather ? p.gather[g] / p.gather_div : g;
      base = p.A + (size_t)srow * p.lda;
    } else {
      const int rb = row - BM;
      const int nb = rb / BN;
      const int n = min(n0 + (rb - nb * BN), p.N - 1);
      base = ((DUAL && nb) ? p.B1 : p.B0) + (size_t)expert * p.b_expert_stride + (size_t)n * p.ldb;
    }
    src[j] = base + kb + ch * 8;
  }

#define AFLEX_GEMM_ISSUE(SM, KT)                                                          \
  do {                                                                                   \
    const int ko_ = min(KT, nk - 1) * BK;                                                \
    _Pragma("unroll") for (int j = 0; j < IPW; ++j)                                      \
        lds_dma16(src[j] + ko_, lds_offset(SM + (wave + 4 * j) * 512));                  \
  } while (0)

  f32x4 acc[NB][TM][TN];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[nb][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const uint16_t* sm) {
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      const int ch = kk * 4 + qg;  // logical 16-byte chunk this lane feeds
      bf16x8 af[TM], bfr[NB][TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int R = wm * WTM + i * 16 + r;
        af[i] = *reinterpret_cast<const bf16x8*>(&sm[R * BK + ((ch ^ ((R >> 1) & 7)) << 3)]);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int R = BM + nb * BN + wn * WTN + j * 16 + r;
          bfr[nb][j] = *reinterpret_cast<const bf16x8*>(&sm[R * BK + ((ch ^ ((R >> 1) & 7)) << 3)]);
        }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[nb][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[nb][j], acc[nb][i][j], 0, 0, 0);
    }
  };

  // Before reading stage kt: vmcnt((STAGES-2)*IPW) means this wave's loads of
  // kt have landed while the STAGES-2 newer stages may still be in flight; the
  // barrier publishes every wave's loads of kt and frees the buffer read in the
  // previous step, which then receives k-step kt+STAGES-1. Prefetches past the
  // last k-step re-read it (clamped index), so every step issues the same
  // number of loads and the count stays exact.
  constexpr int kWait = (STAGES - 2) * IPW;
  constexpr int kWaitImm = (kWait & 15) | ((kWait >> 4) << 14) | (0x7 << 4) | (0xF << 8);
  if (nk > 0) {
#pragma unroll
    for (int st = 0; st < STAGES - 1; ++st) AFLEX_GEMM_ISSUE(sm[st], st);
    int cur = 0;
    for (int kt = 0; kt < nk; ++kt) {
      __builtin_amdgcn_s_waitcnt(kWaitImm);
      __syncthreads();
      const int nxt = cur == 0 ? STAGES - 1 : cur - 1;  // (kt + STAGES - 1) % STAGES
      AFLEX_GEMM_ISSUE(sm[nxt], kt + STAGES - 1);
      compute(sm[cur]);
      cur = cur + 1 == STAGES ? 0 : cur + 1;
    }
    // no load may still target LDS when the work-group retires
    __builtin_amdgcn_s_waitcnt(0);
  }
#undef AFLEX_GEMM_ISSUE

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
