// bf16 GEMM (B in [K, N] layout) kernels, and the launcher of every GEMM
// variant (the kernels themselves are in kf_gemm_mfma.hpp and, for the
// 128x256 tile, kf_gemm_pp.hpp, instantiated in kf_gemm_pp_*.hip).
#include "kf_gemm_mfma.hpp"

namespace kf {

void launch_gemm_bf16_kn(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  launch_shape<false, false>(p, epi, chain, grid, block, stream);
}

int64_t gemm_pp_tiles(int64_t M, int64_t N) {
  return ((M + gemm_pp_tile_m() - 1) / gemm_pp_tile_m()) * ((N + BN - 1) / BN);
}

hipError_t launch_gemm_mfma(const GemmArgs& args, bool fp8, int epi, int chain, hipStream_t stream, bool b_nk,
                            int pp_workgroups) {
  GemmArgs p = args;
  if (pp_workgroups > 0) {
    if (b_nk) return hipErrorInvalidValue;
    p.tiles_m = (int)((p.M + gemm_pp_tile_m() - 1) / gemm_pp_tile_m());
    p.tiles_n = (int)((p.N + BN - 1) / BN);
    const dim3 grid((unsigned)pp_workgroups), block(NT);
    if (fp8)
      launch_gemm_pp_fp8(p, epi, chain, grid, block, stream);
    else
      launch_gemm_pp_bf16(p, epi, chain, grid, block, stream);
    return hipGetLastError();
  }
  p.tiles_m = (int)((p.M + BM - 1) / BM);
  p.tiles_n = (int)((p.N + BN - 1) / BN);
  if (p.raster_group < 1) p.raster_group = 4;
  const dim3 grid(p.tiles_m * p.tiles_n), block(NT);
  if (fp8) {
    if (b_nk)
      launch_gemm_fp8_nk(p, epi, chain, grid, block, stream);
    else
      launch_gemm_fp8_kn(p, epi, chain, grid, block, stream);
  } else {
    if (b_nk)
      launch_gemm_bf16_nk(p, epi, chain, grid, block, stream);
    else
      launch_gemm_bf16_kn(p, epi, chain, grid, block, stream);
  }
  return hipGetLastError();
}

int gemm_mfma_tile_m() { return BM; }
int gemm_mfma_tile_n() { return BN; }

}  // namespace kf
