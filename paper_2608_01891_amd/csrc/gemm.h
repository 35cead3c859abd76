// bf16 MFMA GEMM C = A . B^T for the FFN contractions, gfx950.
//
// A [rows, K] holds tokens (optionally gathered through an index list, which
// is how the MoE reads its token-permuted input without materialising it),
// B [N, K] holds weights in the [out_features, in_features] layout, so both
// operands have the contraction index contiguous and every MFMA operand is
// one 16-byte LDS read. Tiles of BM x BN x 64 stream from HBM straight into a
// ring of 2-4 LDS stages (global_load_lds_dwordx4, no register staging), so
// the loads of the next k-steps are in flight while kt is multiplied
// (v_mfma_f32_16x16x32_bf16 for the 32/64-row tiles, v_mfma_f32_32x32x16_bf16
// for the 128/256-row ones). At decode batch sizes these GEMMs stream
// weights, so the depth of the load pipeline, not the MFMA rate, sets their
// speed.
//
// Variants (template flags):
//   NT_B    weight (B) tile loads are non-temporal.
//   DUAL    two weight matrices (gate, up) share the A tile; the epilogue
//           applies SiLU(gate) * up and stores bf16 (the fused SwiGLU step).
//   OUT_F32 store the fp32 accumulator into split-K partials (one slice per
//           split; a later kernel sums the slices in a fixed order).
//   neither store bf16 (plus an optional bf16 residual, one rounding).
//
// Work decomposition: a 1-D grid over (m-tile, n-tile, k-split). Work-groups
// are dispatched round-robin over the 8 XCDs; the logical tile index is
// remapped so that consecutive tiles (which share an A tile, or for dense
// GEMMs a weight tile across m-tiles) land on the same XCD and its L2. With a
// device-side tile map the remap can run over the real tile count instead of
// the grid (mt_major = 2), so the tiles spread evenly over the XCDs.
// m-tiles come either from a dense row count or from a device-side tile map
// of (expert, first row, end row) triples written by the MoE routing kernel;
// work-groups beyond the map's device-side count exit at once, so the grid is
// sized for the worst case without a host synchronisation.
#pragma once
#include <type_traits>

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
  int split_slots;            // > 0 (tile map only): the split count is chosen on the device from the
                              // row-tile count (at most splits) to fill rounds of split_slots work-groups
  int M;                      // dense row count (tile_map == nullptr)
  const int32_t* tile_map;    // [max_mtiles][3] = (expert, row_begin, row_end)
  const int32_t* num_mtiles;  // device count of valid tile_map entries
  int max_mtiles;
  int n_ntiles;
  int mt_major;               // 1: m-tile is the slow index of the tile order; 2: the same over
                              // the device-side row-tile count (tile_map only), spread over the XCDs
  uint16_t* C;                // bf16 output [rows, ldc]
  int ldc;
  const uint16_t* R;          // optional bf16 residual [rows, ldc] added before rounding (plain bf16 output only)
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
  uint32_t saved;  // m0 is reserved to the compiler: restore it after the load
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gptr), "s"(lds_s)
      : "memory");
}

// The same load marked non-temporal: weights that one work-group streams
// exactly once (a 32-row tile covers all of a decode microbatch's rows of an
// expert) need not stay in the caches.
__device__ __forceinline__ void lds_dma16_nt(const void* gptr, uint32_t lds) {
  const uint32_t lds_s = __builtin_amdgcn_readfirstlane(lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off nt\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gptr), "s"(lds_s)
      : "memory");
}

__device__ __forceinline__ int xcd_remap(int w, int nwg) {
  const int q = nwg >> 3, rem = nwg & 7, x = w & 7, j = w >> 3;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + j;
}

// Split-K count for `tiles` output tiles over K = 64 * ksteps: the smallest
// count up to smax whose work-groups fill the rounds of `slots` concurrent
// work-groups they need to at least 90%, else the best-filled one; *kps is the
// k elements per split (a multiple of 64). The device-side twin of the host
// planner, used where the row-tile count is known on the device only.
__device__ __forceinline__ void split_plan_slots(int tiles, int ksteps, int smax, int slots, int* splits, int* kps) {
  int s = 1;
  long long bn = 0, bd = 1;  // best fill so far, bn / bd
  for (int c = 1; c <= smax; ++c) {
    const long long wgs = (long long)tiles * c;
    const long long cap = ((wgs + slots - 1) / slots) * slots;
    if (10 * wgs >= 9 * cap) {
      s = c;
      break;
    }
    if (wgs * bd > bn * cap) {
      bn = wgs;
      bd = cap;
      s = c;
    }
  }
  const int steps = (ksteps + s - 1) / s;
  *splits = (ksteps + steps - 1) / steps;
  *kps = steps * 64;
}

// BM x BN output tile, WM x WN waves (each a (BM/WM) x (BN/WN) sub-tile of
// MS x MS MFMA tiles: v_mfma_f32_16x16x32_bf16 or v_mfma_f32_32x32x16_bf16),
// BK-wide k-steps, LDS_BYTES of LDS per work-group (the ring has as many
// stages as fit; 80 KiB lets two work-groups share a CU). The 32x32 MFMA
// sustains a higher issue rate and serves the MFMA-bound tiles.
template <int BM, int BN, int WM, int WN, int BK, int MS, bool DUAL, bool OUT_F32, int LDS_BYTES, bool NT_B = false>
__global__ __launch_bounds__(64 * WM * WN, LDS_BYTES > 81920 ? 1 : 2) void gemm_nt_kernel(GemmParams p) {
  constexpr int NW = WM * WN;
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / MS, TN = WTN / MS;
  using Acc = typename std::conditional<MS == 16, f32x4, f32x16>::type;
  constexpr int NACC = MS == 16 ? 4 : 16;
  constexpr int CPR = BK / 8;           // 16-byte chunks per LDS row
  constexpr int WIN = 128 / BK;         // rows per 256-byte bank window
  constexpr int ROWS = BM + NB * BN;    // LDS rows per stage: A tile, then the B tile(s)
  constexpr int INS = ROWS * CPR / 64;  // 1 KiB wave-loads per stage
  constexpr int IPW = INS / NW;         // per wave
  constexpr int STAGE_BYTES = ROWS * BK * 2;
  constexpr int STAGES = LDS_BYTES / STAGE_BYTES;
  static_assert(BK == 32 || BK == 64, "k-step");
  static_assert(MS == 16 || MS == 32, "MFMA shape");
  static_assert(TM >= 1 && TN >= 1 && INS % NW == 0, "tile shape");
  static_assert(STAGES >= 2 && (STAGES - 2) * IPW < 64, "stages");

  // Ring of STAGES buffers filled by direct global->LDS loads: lane l of a
  // wave-load writes the 16 bytes at slot base + l. Slot s of a stage holds
  // row s / CPR, 16-byte chunk (s % CPR) ^ swz(row) of the tile, with
  // swz(row) = (row / WIN) % CPR, so the 16 rows of an MFMA fragment read fall
  // on distinct bank groups.
  __shared__ __attribute__((aligned(16))) uint16_t sm[STAGES][ROWS * BK];

  int t, splits = p.splits, kps = p.k_per_split, mrange = p.max_mtiles;
  if (p.mt_major == 2 || p.split_slots > 0) {
    // Row tiles from the device-side count (and the split count planned from
    // it): the real tiles spread evenly over the XCDs. Expert-major
    // (mt_major = 2), each XCD takes consecutive n-tiles of one or two experts,
    // whose token rows then stay in its L2.
    const int mtiles = *p.num_mtiles;
    if (p.split_slots > 0) split_plan_slots(mtiles * p.n_ntiles, p.K / 64, p.splits, p.split_slots, &splits, &kps);
    const int nreal = mtiles * p.n_ntiles * splits;
    if ((int)blockIdx.x >= nreal) return;
    t = xcd_remap(blockIdx.x, nreal);
    mrange = mtiles;
  } else {
    t = xcd_remap(blockIdx.x, gridDim.x);
  }
  const int split = t % splits;
  const int rest = t / splits;
  int mt, nt;
  if (p.mt_major) {
    nt = rest % p.n_ntiles;
    mt = rest / p.n_ntiles;
  } else if (p.tile_map == nullptr && p.max_mtiles > 8) {
    // Dense GEMMs with many row tiles: groups of 8 row tiles, row fastest, so
    // the 32 work-groups an XCD runs at a time cover 8 A tiles x 4 weight tiles
    // (12 tile streams through its L2 instead of 16 + 2).
    const int per = 8 * p.n_ntiles, grp = rest / per, in = rest - grp * per;
    const int gm = min(8, p.max_mtiles - grp * 8);
    mt = grp * 8 + in % gm;
    nt = in / gm;
  } else {
    mt = rest % mrange;
    nt = rest / mrange;
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
  const int kb = split * kps;
  const int ke = min(p.K, kb + kps);
  const int nk = (ke - kb) / BK;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  // MFMA operand lane roles: row/column r of the tile, k-slice g (8 wide).
  const int r = lane & (MS - 1), qg = lane / MS;
  const int wm = wave / WN, wn = wave % WN;

  // Global source of each of this lane's wave-loads (fixed over k). Rows past
  // the tile (A rows >= row1, weight rows >= N) read a valid row instead; their
  // products land in output rows/columns that are never stored.
  const uint16_t* src[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int slot = (wave + NW * j) * 64 + lane;
    const int row = slot / CPR;
    const int ch = (slot % CPR) ^ ((row / WIN) % CPR);
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
        if (NT_B && ((wave + NW * j) * 64) / CPR >= BM)                                    \
          lds_dma16_nt(src[j] + ko_, lds_offset(SM + (wave + NW * j) * 512));              \
        else                                                                             \
          lds_dma16(src[j] + ko_, lds_offset(SM + (wave + NW * j) * 512));                 \
  } while (0)

  Acc acc[NB][TM][TN];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < NACC; ++e) acc[nb][i][j][e] = 0.f;

  constexpr int KC = MS == 16 ? 32 : 16;  // k per MFMA
  constexpr int CPS = BK / KC;             // MFMA k-chunks per stage
  const int nchunks = nk * CPS;

  // Fragments of k-chunk C (of stage C / CPS) into registers FA (the first
  // TMA row blocks of the wave) and FB.
#define AFLEX_GEMM_READ(FA, FB, C, TMA)                                                    \
  do {                                                                                    \
    const int kt_ = (C) / CPS;                                                            \
    const uint16_t* smp_ = sm[kt_ % STAGES];                                              \
    const int ch_ = ((C) - kt_ * CPS) * (KC / 8) + qg;                                    \
    _Pragma("unroll") for (int i = 0; i < (TMA); ++i) {                                   \
      const int R = wm * WTM + i * MS + r;                                                \
      FA[i] = *reinterpret_cast<const bf16x8*>(&smp_[R * BK + ((ch_ ^ ((R / WIN) % CPR)) << 3)]); \
    }                                                                                     \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb)                                     \
        _Pragma("unroll") for (int j = 0; j < TN; ++j) {                                  \
      const int R = BM + nb * BN + wn * WTN + j * MS + r;                                 \
      FB[nb][j] = *reinterpret_cast<const bf16x8*>(&smp_[R * BK + ((ch_ ^ ((R / WIN) % CPR)) << 3)]); \
    }                                                                                     \
  } while (0)
#define AFLEX_GEMM_MMA(FA, FB, TMA)                                                        \
  do {                                                                                    \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb)                                     \
        _Pragma("unroll") for (int i = 0; i < (TMA); ++i)                                 \
            _Pragma("unroll") for (int j = 0; j < TN; ++j) {                              \
      if constexpr (MS == 16)                                                             \
        acc[nb][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(FA[i], FB[nb][j], acc[nb][i][j], 0, 0, 0); \
      else                                                                                \
        acc[nb][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(FA[i], FB[nb][j], acc[nb][i][j], 0, 0, 0); \
    }                                                                                     \
  } while (0)
  // Make stage KT1 readable: vmcnt((STAGES-2)*IPW) means this wave's loads of
  // KT1 have landed while the STAGES-2 newer stages may still be in flight; the
  // barrier (which first drains this wave's LDS reads) publishes every wave's
  // loads of KT1 and guarantees stage KT1-1 is no longer read, so its buffer
  // receives k-step KT1+STAGES-1. Prefetches past the last k-step re-read it
  // (clamped index), so every stage issues the same number of loads and the
  // count stays exact.
  constexpr int kWait = (STAGES - 2) * IPW;
  constexpr int kWaitImm = (kWait & 15) | ((kWait >> 4) << 14) | (0x7 << 4) | (0xF << 8);
#define AFLEX_GEMM_STAGE(KT1)                                                              \
  do {                                                                                    \
    __builtin_amdgcn_s_waitcnt(kWaitImm);                                                 \
    __syncthreads();                                                                      \
    AFLEX_GEMM_ISSUE(sm[((KT1) + STAGES - 1) % STAGES], (KT1) + STAGES - 1);              \
  } while (0)

  // Row blocks of this wave that hold rows of the tile: a partly filled row
  // tile (an expert's last rows, a dense remainder) multiplies only those.
  const int nact = (min(max(row1 - row0 - wm * WTM, 0), WTM) + MS - 1) / MS;
  if (nk > 0 && nact == 0) {
    // No row of this wave lies in the tile: it multiplies nothing, but still
    // loads its share of every stage and takes part in the same barriers, so
    // the MFMA pipe of its SIMD is left to the other wave.
#pragma unroll
    for (int st = 0; st < STAGES - 1; ++st) AFLEX_GEMM_ISSUE(sm[st], st);
    AFLEX_GEMM_STAGE(0);
    for (int kt = 0; kt < nk; ++kt) AFLEX_GEMM_STAGE(kt + 1);
    __builtin_amdgcn_s_waitcnt(0);
  } else if (nk > 0) {
    // Software pipeline over k-chunks (an even number per stage):
    // the fragment reads of chunk c+1 are interleaved one by one with the MFMAs
    // of chunk c (the wave issues in order, so a read placed between two MFMAs
    // goes out while the first executes); the stage wait and barrier follow,
    // then the reads of chunk c+2 interleaved with the MFMAs of chunk c+1. The
    // body has no data-dependent guards, so the only LDS waits are for reads
    // issued a chunk earlier; the last iteration's stage step and read of
    // chunk c+2 re-read the last k-step (clamped), which is never used.
    // Measured against the guarded two-chunk loop (whose waits covered the
    // reads just issued): 4-5% at the MFMA-bound shapes, bit-identical.
    auto kloop = [&](auto tma) {
      constexpr int TMA = decltype(tma)::value;
      bf16x8 fa0[TMA], fb0[NB][TN], fa1[TMA], fb1[NB][TN];
#pragma unroll
      for (int st = 0; st < STAGES - 1; ++st) AFLEX_GEMM_ISSUE(sm[st], st);
      AFLEX_GEMM_STAGE(0);
      AFLEX_GEMM_READ(fa0, fb0, 0, TMA);
      static_assert(CPS % 2 == 0, "an even number of MFMA k-chunks per stage");
      // One MFMA, one fragment read, alternately, then whichever kind remains.
      constexpr int NREAD = TMA + NB * TN, NMMA = NB * TMA * TN;
      constexpr int NPAIR = NREAD < NMMA ? NREAD : NMMA;
#define AFLEX_GEMM_INTERLEAVE()                                                              \
  do {                                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < NPAIR; ++i_) {                                   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0); /* one MFMA */                     \
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); /* one LDS read */                 \
    }                                                                                        \
    if constexpr (NMMA > NREAD) __builtin_amdgcn_sched_group_barrier(0x008, NMMA - NREAD, 0); \
    if constexpr (NREAD > NMMA) __builtin_amdgcn_sched_group_barrier(0x100, NREAD - NMMA, 0); \
    __builtin_amdgcn_sched_barrier(0);                                                       \
  } while (0)
      for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
        for (int cc = 0; cc < CPS; cc += 2) {
          const int c = kt * CPS + cc;
          AFLEX_GEMM_READ(fa1, fb1, c + 1, TMA);
          AFLEX_GEMM_MMA(fa0, fb0, TMA);
          AFLEX_GEMM_INTERLEAVE();
          if (cc + 2 == CPS) {
            AFLEX_GEMM_STAGE(kt + 1);
            __builtin_amdgcn_sched_barrier(0);
          }
          AFLEX_GEMM_READ(fa0, fb0, min(c + 2, nchunks - 1), TMA);
          AFLEX_GEMM_MMA(fa1, fb1, TMA);
          AFLEX_GEMM_INTERLEAVE();
        }
      }
#undef AFLEX_GEMM_INTERLEAVE
      // no load may still target LDS when the work-group retires
      __builtin_amdgcn_s_waitcnt(0);
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2 <= TM ? 2 : TM>;
    using I3 = std::integral_constant<int, 3 <= TM ? 3 : TM>;
    using I4 = std::integral_constant<int, 4 <= TM ? 4 : TM>;
    using IT = std::integral_constant<int, TM>;
    static_assert(TM <= 5, "row blocks per wave");
    if (nact == 1)
      kloop(I1{});
    else if (nact == 2)
      kloop(I2{});
    else if (nact == 3)
      kloop(I3{});
    else if (nact == 4 || TM == 4)
      kloop(I4{});
    else
      kloop(IT{});
  }
#undef AFLEX_GEMM_READ
#undef AFLEX_GEMM_MMA
#undef AFLEX_GEMM_STAGE
#undef AFLEX_GEMM_ISSUE

  // Epilogue. 16x16 tiles: accumulator e of a lane is row 4 g + e, column r.
  // 32x32 tiles: row (e / 4) * 8 + 4 g + e % 4, column r.
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * WTN + j * MS + r;
      if (col >= p.N) continue;
#pragma unroll
      for (int e = 0; e < NACC; ++e) {
        const int er = MS == 16 ? 4 * qg + e : (e >> 2) * 8 + 4 * qg + (e & 3);
        const int row = row0 + wm * WTM + i * MS + er;
        if (row >= row1) continue;
        if (OUT_F32) {
          p.P[(size_t)split * p.p_split_stride + (size_t)row * p.ldp + col] = acc[0][i][j][e];
        } else if (DUAL) {
          const float g = acc[0][i][j][e];
          const float u = acc[NB - 1][i][j][e];
          const float h = g / (1.f + __expf(-g)) * u;
          p.C[(size_t)row * p.ldc + col] = f2bf(h);
        } else {
          const float r = p.R ? bf2f(p.R[(size_t)row * p.ldc + col]) : 0.f;
          p.C[(size_t)row * p.ldc + col] = f2bf(acc[0][i][j][e] + r);
        }
      }
    }
  }
}

}  // namespace aflex
