// OCP fp8 e4m3 GEMM, B in [K, N] layout, two workgroups per CU: the
// instantiations of the kernel in kf_gemm_pp.hpp.
#include "kf_gemm_pp.hpp"

namespace kf {

void launch_gemm_pp_fp8(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  pp_launch_shape<true>(p, epi, chain, grid, block, stream);
}

}  // namespace kf
