// bf16 GEMM, B in [K, N] layout, two workgroups per CU: the instantiations of
// the kernel in kf_gemm_pp.hpp.
#include "kf_gemm_pp.hpp"

namespace kf {

void launch_gemm_pp_bf16(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  pp_launch_shape<false>(p, epi, chain, grid, block, stream);
}

int gemm_pp_tile_m() { return kPpBM; }

}  // namespace kf
