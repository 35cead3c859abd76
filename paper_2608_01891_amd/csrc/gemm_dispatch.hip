// Instantiations of the FFN GEMM tiles and their launch helpers.
//
// Row-tile size selects the shape: 32- and 64-row tiles stream weights (4
// waves, 16x16x32 MFMA, 64-wide k-steps, two work-groups per CU, HBM-bound);
// 128-, 256- and 320-row tiles are the 8-wave 32x32x16 MFMA shapes (wave
// tiles of 64, 128 or 160 rows by 32 columns of each gate/up matrix or 64
// columns of the down matrix, one work-group per CU in the whole 160 KiB of
// LDS; the 320-row tiles take 240 registers, still two waves per SIMD). Both take
// 64-wide k-steps, so every k-step reads whole 128-byte lines of each row: a
// ring of three stages for the 128-row tiles, two (the next k-step loads
// while the current one is multiplied) for the 256-row tiles, which was
// faster than five stages of 32-wide k-steps (dense T = 512: 474 -> 432 us,
// T = 4096: 3.02 -> 2.82 ms). Weights that one tile streams
// exactly once load non-temporally: always for 32-row tiles, for 64- and
// 128-row tiles when the caller has a single row tile per weight matrix
// (measured on the 128-row tiles, dense T = 128: 215 -> 188 us for the
// 64-wide k-steps, 175 us with non-temporal loads; with 32-wide k-steps
// non-temporal loads were slower, the second half of each line then coming
// from HBM again).
#include "ffn_plan.h"
#include "profile.h"

namespace aflex {

template <int BM, int BN, int WM, int WN, int BK, int MS, bool DUAL, bool F32, int LDS, bool NT = false>
static void go(const GemmParams& g, unsigned grid, hipStream_t stream) {
  gemm_nt_kernel<BM, BN, WM, WN, BK, MS, DUAL, F32, LDS, NT><<<grid, 64 * WM * WN, 0, stream>>>(g);
}

static unsigned grid_of(const GemmParams& g) {
  return (unsigned)((long long)g.max_mtiles * g.n_ntiles * g.splits);
}

hipError_t launch_gate_up(int bm, bool once, const GemmParams& g, hipStream_t stream) {
  const unsigned grid = grid_of(g);
  if (grid == 0) return hipSuccess;
  ProfScope ps("gemm_gate_up", stream);
  switch (bm) {
    case 32: go<32, 64, 1, 4, 64, 16, true, false, 81920, true>(g, grid, stream); break;
    case 64:
      if (once)
        go<64, 64, 2, 2, 64, 16, true, false, 81920, true>(g, grid, stream);
      else
        go<64, 64, 2, 2, 64, 16, true, false, 81920>(g, grid, stream);
      break;
    case 128:
      if (once)
        go<128, 128, 2, 4, 64, 32, true, false, 163840, true>(g, grid, stream);
      else
        go<128, 128, 2, 4, 64, 32, true, false, 163840>(g, grid, stream);
      break;
    case 320: go<320, 128, 2, 4, 64, 32, true, false, 163840>(g, grid, stream); break;
    default: go<256, 128, 2, 4, 64, 32, true, false, 163840>(g, grid, stream); break;
  }
  return hipGetLastError();
}

template <bool F32>
static void down(int bm, bool once, const GemmParams& g, unsigned grid, hipStream_t stream) {
  switch (bm) {
    case 32: go<32, 128, 1, 4, 64, 16, false, F32, 81920, true>(g, grid, stream); break;
    case 64:
      if (once)
        go<64, 128, 2, 2, 64, 16, false, F32, 81920, true>(g, grid, stream);
      else
        go<64, 128, 2, 2, 64, 16, false, F32, 81920>(g, grid, stream);
      break;
    case 128:
      if (once)
        go<128, 256, 2, 4, 64, 32, false, F32, 163840, true>(g, grid, stream);
      else
        go<128, 256, 2, 4, 64, 32, false, F32, 163840>(g, grid, stream);
      break;
    case 320: go<320, 256, 2, 4, 64, 32, false, F32, 163840>(g, grid, stream); break;
    default: go<256, 256, 2, 4, 64, 32, false, F32, 163840>(g, grid, stream); break;
  }
}

hipError_t launch_down(int bm, bool f32_partials, bool once, const GemmParams& g, hipStream_t stream) {
  const unsigned grid = grid_of(g);
  if (grid == 0) return hipSuccess;
  ProfScope ps("gemm_down", stream);
  if (f32_partials)
    down<true>(bm, once, g, grid, stream);
  else
    down<false>(bm, once, g, grid, stream);
  return hipGetLastError();
}

}  // namespace aflex
