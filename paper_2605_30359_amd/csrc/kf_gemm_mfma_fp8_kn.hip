// OCP fp8 e4m3 GEMM, B in [K, N] layout: the instantiations of the kernel in kf_gemm_mfma.hpp.
#include "kf_gemm_mfma.hpp"

namespace kf {

void launch_gemm_fp8_kn(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  launch_shape<true, false>(p, epi, chain, grid, block, stream);
}

}  // namespace kf
