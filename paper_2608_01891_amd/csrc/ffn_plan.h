// Tile and split-K planning shared by the dense and MoE FFN launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>

#include "gemm.h"

namespace aflex {

// Output columns per gate/up tile (x2 weight rows) and per down tile. The
// 128- and 256-row tiles are the 8-wave 32x32x16 MFMA shapes (one work-group
// per CU); dense GEMMs take 128-row tiles for 33 ... 128 tokens (measured:
// T = 128 262 -> 211 us against 256-row tiles).
inline int gate_bn(int bm) { return bm >= 128 ? 128 : 64; }

inline int down_bn(int bm) { return bm >= 128 ? 256 : 128; }
// Work-groups the down GEMM's split-K aims for: the 256-row tiles run one
// work-group per CU, so one round of the chip; smaller tiles two per CU.
constexpr int kOneWgPerCuTarget = 256;
inline int down_target(int bm) { return bm >= 128 ? kOneWgPerCuTarget : (bm == 64 ? 2048 : 512); }
// Work-groups resident on the 256 CUs at once: one per CU for the 8-wave
// tiles (the whole LDS), two for the 4-wave tiles.
inline int concurrent_wgs(int bm) { return bm >= 128 ? 256 : 512; }

struct FfnPlan {
  int bm;           // rows per m-tile: 32, 64, 128 or 256
  int down_splits;  // split-K factor of the down GEMM
  int down_kps;     // k elements per split (multiple of 64)
};

// Rows per m-tile for grouped GEMMs with the given average rows per expert.
// Up to 32 rows a tile covers a typical expert (its weights are streamed once,
// non-temporally); up to 48 rows 64-row tiles, two work-groups per CU (an
// expert's second tile re-reads its weights from L2; at 32 rows per expert
// 535 us against 611 us with 128-row tiles); up to 144 rows the 8-wave
// 128-row tile; beyond, the 256-row shape (Mixtral shapes, 128 rows per
// expert: 828 us with 128-row tiles, 857 with 256; 160 rows: 936 and 888).
//
// Above 144 rows the tile is 256 or 320 rows, whichever covers an expert two
// standard deviations above the average (routing counts spread about as a
// binomial, sigma ~ sqrt(average)) with fewer row tiles; ties go to 256. An
// expert just over a multiple of 256 rows would otherwise pay a nearly empty
// tile that streams all of its weights again (Mixtral T = 2048: 472-541 rows
// per expert, 21 row tiles of 256 against 16 of 320).
inline int pick_bm(double rows_per_expert) {
  if (rows_per_expert * 1.3 <= 32) return 32;
  if (rows_per_expert <= 48) return 64;
  if (rows_per_expert <= 144) return 128;
  const double hi = rows_per_expert + 2.0 * sqrt(rows_per_expert);
  return ceil(hi / 320.0) < ceil(hi / 256.0) ? 320 : 256;
}

// Split K of the down GEMM, keeping at least `min_steps` 64-wide k-steps per
// split. With `slots` > 0 (the tile count is exact: dense GEMMs, and the
// one-work-group-per-CU tiles) the split count is the smallest whose
// work-groups fill the rounds of `slots` concurrent work-groups they need to
// at least 90% (measured best for the dense down GEMM at T = 256 ... 4096:
// 12, 6, 3, 3-4 splits; a nearly empty last round leaves a few work-groups
// streaming alone at the end); more splits only add fp32 partials to reduce.
// Otherwise (a worst-case tile count) about `target` work-groups.
inline void plan_splits(int base_tiles, int K, int target, int slots, int min_steps, int* splits, int* kps) {
  const int ksteps = K / 64;
  int smax = ksteps / min_steps;
  if (smax < 1) smax = 1;
  int s = (target + base_tiles - 1) / base_tiles;
  if (slots > 0) {
    double best_u = 0.0;
    for (int c = 1; c <= smax && c <= 64; ++c) {
      const long long wgs = (long long)base_tiles * c;
      const double u = (double)wgs / (double)(((wgs + slots - 1) / slots) * slots);
      if (u >= 0.9) {
        s = c;
        break;
      }
      if (u > best_u + 1e-9) {
        best_u = u;
        s = c;
      }
    }
  }
  if (s > smax) s = smax;
  if (s < 1) s = 1;
  const int steps = (ksteps + s - 1) / s;
  *splits = (ksteps + steps - 1) / steps;
  *kps = steps * 64;
}

inline FfnPlan plan_dense(int T, int H, int I) {
  FfnPlan pl;
  pl.bm = T <= 32 ? 32 : (T <= 128 ? 128 : 256);
  const int mtiles = (T + pl.bm - 1) / pl.bm;
  const int ntiles = (H + down_bn(pl.bm) - 1) / down_bn(pl.bm);
  plan_splits(mtiles * ntiles, I, down_target(pl.bm), concurrent_wgs(pl.bm), 8, &pl.down_splits, &pl.down_kps);
  return pl;
}

// `once`: the call has (dense) or is expected to have (MoE, from the average
// rows per expert) a single row tile per weight matrix, so every weight byte
// is read once and its loads can be non-temporal.
hipError_t launch_gate_up(int bm, bool once, const GemmParams& g, hipStream_t stream);
hipError_t launch_down(int bm, bool f32_partials, bool once, const GemmParams& g, hipStream_t stream);

}  // namespace aflex
