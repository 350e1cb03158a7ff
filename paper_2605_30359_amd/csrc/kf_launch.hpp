// Host-side launchers of the kernels of libkf.so (one per kernel family).
// Each enqueues its kernel(s) on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>

#include "kf_internal.hpp"

namespace kf {

// bf16 GEMM + epilogue; `epi` is an EpiShape.
hipError_t launch_gemm_bf16(const GemmArgs& args, int epi, hipStream_t stream, bool b_nk);
int gemm_bf16_tile_m();
int gemm_bf16_tile_n();

// fp32 GEMM + element-wise epilogue.
hipError_t launch_gemm_f32(const GemmArgs& args, bool b_nk, hipStream_t stream);

// Row softmax rescale / logsumexp combine from per-tile partials.
hipError_t launch_row_finish(bool softmax, const void* partials, int tiles, int64_t M, int64_t N, void* out,
                             int64_t ldo, bool out_bf16, hipStream_t stream);
int row_finish_max_tiles();

}  // namespace kf
