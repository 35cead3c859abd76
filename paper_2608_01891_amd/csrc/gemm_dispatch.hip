// Instantiations of the FFN GEMM tiles and their launch helpers.
#include "ffn_plan.h"
#include "profile.h"

namespace aflex {

static unsigned grid_of(const GemmParams& g) {
  return (unsigned)((long long)g.max_mtiles * g.n_ntiles * g.splits);
}

hipError_t launch_gate_up(int bm, const GemmParams& g, hipStream_t stream) {
  const unsigned grid = grid_of(g);
  if (grid == 0) return hipSuccess;
  ProfScope ps("gemm_gate_up", stream);
  switch (bm) {
    case 32: gemm_nt_kernel<32, kGateBN, 1, 4, true, false><<<grid, 256, 0, stream>>>(g); break;
    case 64: gemm_nt_kernel<64, kGateBN, 2, 2, true, false><<<grid, 256, 0, stream>>>(g); break;
    default: gemm_nt_kernel<128, kGateBN, 2, 2, true, false><<<grid, 256, 0, stream>>>(g); break;
  }
  return hipGetLastError();
}

hipError_t launch_down(int bm, bool f32_partials, const GemmParams& g, hipStream_t stream) {
  const unsigned grid = grid_of(g);
  if (grid == 0) return hipSuccess;
  ProfScope ps("gemm_down", stream);
  if (f32_partials) {
    switch (bm) {
      case 32: gemm_nt_kernel<32, 128, 1, 4, false, true><<<grid, 256, 0, stream>>>(g); break;
      case 64: gemm_nt_kernel<64, 128, 2, 2, false, true><<<grid, 256, 0, stream>>>(g); break;
      default: gemm_nt_kernel<128, 128, 2, 2, false, true><<<grid, 256, 0, stream>>>(g); break;
    }
  } else {
    switch (bm) {
      case 32: gemm_nt_kernel<32, 128, 1, 4, false, false><<<grid, 256, 0, stream>>>(g); break;
      case 64: gemm_nt_kernel<64, 128, 2, 2, false, false><<<grid, 256, 0, stream>>>(g); break;
      default: gemm_nt_kernel<128, 128, 2, 2, false, false><<<grid, 256, 0, stream>>>(g); break;
    }
  }
  return hipGetLastError();
}

}  // namespace aflex
