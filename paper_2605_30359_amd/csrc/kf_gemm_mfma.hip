// bf16 GEMM (B in [K, N] layout) kernels, and the launcher of every GEMM
// variant (the kernel itself is in kf_gemm_mfma.hpp).
#include "kf_gemm_mfma.hpp"

namespace kf {

void launch_gemm_bf16_kn(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  launch_shape<false, false>(p, epi, chain, grid, block, stream);
}

hipError_t launch_gemm_mfma(const GemmArgs& args, bool fp8, int epi, int chain, hipStream_t stream, bool b_nk) {
  GemmArgs p = args;
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
