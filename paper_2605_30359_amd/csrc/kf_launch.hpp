// Host-side launchers of the kernels of libkf.so (one per kernel family).
// Each enqueues its kernel(s) on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>

#include "kf_internal.hpp"

namespace kf {

// Workgroups of `kernel` (block threads, no dynamic LDS) that the device holds
// at once: compute units x resident workgroups per compute unit.  Streaming
// kernels size a grid-stride launch by it, so that no partly filled last
// round of workgroups trails the launch.  Callers cache it per kernel.
template <typename Kernel>
inline int resident_blocks(Kernel kernel, int block) {
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, block, 0) != hipSuccess) {
    (void)hipGetLastError();
    return 1024;
  }
  return (cus > 0 ? cus : 1) * (per > 0 ? per : 1);
}

// Device address of the static scratch array on `device` (the current
// device), looked up on the first call per device; scratch_bytes() is its
// size.
hipError_t scratch_address(int device, void** out);
size_t scratch_bytes();

// bf16 or OCP fp8 e4m3 GEMM + epilogue on the matrix cores; `epi` is an
// EpiShape, `chain` a compile-time chain id (0: the op list is interpreted).
// pp_workgroups == 0 runs the 256x256 tile kernel; > 0 the 128x256 kernel
// with two workgroups per CU (B in KN layout only) as a persistent grid of
// that many workgroups.
hipError_t launch_gemm_mfma(const GemmArgs& args, bool fp8, int epi, int chain, hipStream_t stream, bool b_nk,
                            int pp_workgroups);
// Tiles of the 128x256 kernel for an M x N output.
int64_t gemm_pp_tiles(int64_t M, int64_t N);
int gemm_mfma_tile_m();
int gemm_mfma_tile_n();

// Row-wise op chain with no contraction (h = A), one workgroup per row;
// N <= rowwise_max_cols(); `chain` as for the GEMM (0: interpreted).
hipError_t launch_rowwise(const RowArgs& args, int chain, hipStream_t stream);
int rowwise_max_cols();
// True for op lists that end with a row logsumexp or cross-entropy after
// element-wise ops and a bias only: launch_rowwise streams those rows, any
// N (a multiple of 8).
bool row_reduce_streams(const EpiProgram& prog);
// The kernel launch_rowwise runs for an op list (GroupNorm group width
// `gn_group` columns, 0 if none).
const char* rowwise_kernel(const EpiProgram& prog, int gn_group);

// The matrix-core rate probe: `workgroups` workgroups of probe_threads()
// threads, each SIMD issuing `iters` rounds of 8 independent 32x32 MFMAs
// (bf16 32x32x16 or fp8 32x32x64) from registers; sink takes one float per
// thread, stamps 4 per workgroup (shader-clock counter at start and end,
// constant-rate counter at start and end).
hipError_t launch_mfma_probe(bool fp8, int64_t iters, int workgroups, float* sink, long long* stamps,
                             hipStream_t stream);
int probe_threads();
// The copy probe: dst[i] = src[i] over `chunks` 16-byte chunks (streaming
// stores), a resident-sized grid-stride launch.
hipError_t launch_copy_probe(const void* src, void* dst, int64_t chunks, hipStream_t stream);

// fp32 GEMM + element-wise epilogue.
hipError_t launch_gemm_f32(const GemmArgs& args, bool b_nk, hipStream_t stream);

// Row softmax rescale / logsumexp combine from per-tile partials; with
// `targets`, the cross-entropy logsumexp - tlogit[m] (NaN where a target is
// outside [0, N)).
hipError_t launch_row_finish(bool softmax, const void* partials, int tiles, int64_t M, int64_t N, void* out,
                             int64_t ldo, bool out_bf16, hipStream_t stream, const int32_t* targets = nullptr,
                             const float* tlogit = nullptr);
int row_finish_max_tiles();

}  // namespace kf

namespace kf {

// 3x3 conv (bf16, NCHW/OIHW) + fused element-wise ops and 2x2 max-pool:
// launch_conv_pack repacks the weights into `packed_weights` (device scratch
// of 9 * cout * cin bf16, layout [tap][co][ci]), launch_conv_bf16 runs the
// convolution from it.  Supports cin == conv_bf16_cin(), width ==
// conv_bf16_width(), cout == conv_bf16_cout(), even height.
hipError_t launch_conv_pack(const ConvArgs& args, void* packed_weights, hipStream_t stream);
hipError_t launch_conv_bf16(const ConvArgs& args, const void* packed_weights, int chain, hipStream_t stream);
int conv_bf16_cin();
int conv_bf16_width();
int conv_bf16_cout();
// The general conv (ConvArgs.variant 2): any shape; its packed weights hold
// 9 * cout * conv_gen_cin_pad(cin) bf16 and it launches conv_gen_tiles(...)
// workgroups.
__host__ __device__ int conv_gen_cin_pad(int cin);
int64_t conv_gen_tiles(int64_t batch, int64_t H, int64_t W, int64_t cout);

// 3x3x3 conv (bf16, channels-last input, OIDHW weight) + fused bias,
// element-wise ops, channel softmax and two 3-D max-pools:
// launch_conv3d_pack repacks the weights into `packed_weights` (device
// scratch of conv3d_packed_bytes()), launch_conv3d_bf16 runs the convolution
// from it.  Supports cin == conv3d_cin(), cout == conv3d_cout().
hipError_t launch_conv3d_pack(const void* w, void* packed_weights, hipStream_t stream);
hipError_t launch_conv3d_bf16(const Conv3dArgs& args, const void* packed_weights, int chain, hipStream_t stream);
int conv3d_cin();
int conv3d_cout();
size_t conv3d_packed_bytes();

// The general 3x3x3 conv (any batch, cin, cout, D, H, W >= 3) + bias and
// element-wise ops, reading the input through its element strides (NCDHW or
// channels-last), writing NCDHW; launch_conv3d_gen_pack repacks the OIDHW
// weights into `packed` (conv3d_gen_packed_bytes()), launch_conv3d_gen runs
// conv3d_gen_tiles(...) workgroups (fewer than 2^31).
struct Conv3dGenArgs {
  const void* x;                      // input [batch, cin, D, H, W] at these element strides
  int64_t sn, sc, sd, sh, sw;
  int32_t batch, cin, cout, D, H, W;
  EpiProgram prog;                    // BIAS and element-wise ops
  const float* bias;                  // [cout] or null
  void* out;                          // [batch, cout, D - 2, H - 2, W - 2] contiguous
};
hipError_t launch_conv3d_gen_pack(const void* w, void* packed, int cout, int cin, hipStream_t stream);
hipError_t launch_conv3d_gen(const Conv3dGenArgs& args, const void* packed, hipStream_t stream);
int64_t conv3d_gen_tiles(int64_t batch, int64_t D, int64_t H, int64_t W, int64_t cout);
size_t conv3d_gen_packed_bytes(int64_t cout, int64_t cin);

}  // namespace kf

namespace kf {

// Unfused comparator kernels (one per op, memory-bound).  `fdiv` / `fmod`
// map a flat element index to its feature for BIAS: (i / fdiv) % fmod.
hipError_t launch_unfused_elementwise(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t n, int kind,
                                      float p0, float p1, const float* bias, int64_t fdiv, int64_t fmod,
                                      hipStream_t stream);
hipError_t launch_unfused_residual(const void* in, bool in_bf16, const void* res, bool res_bf16, void* out,
                                   bool out_bf16, int64_t n, hipStream_t stream);
hipError_t launch_unfused_groupnorm(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                    int groups, float eps, const float* gamma, const float* beta, hipStream_t stream);
// kind: KF_OP_ROW_SOFTMAX, _LOGSUMEXP or _CROSS_ENTROPY (with targets)
hipError_t launch_unfused_rowop(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                int kind, const int32_t* targets, hipStream_t stream);
hipError_t launch_unfused_maxpool(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int H,
                                  int W, hipStream_t stream);
hipError_t launch_unfused_channel_softmax(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t batch,
                                         int channels, int64_t spatial, hipStream_t stream);
hipError_t launch_unfused_maxpool3d(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int D,
                                    int H, int W, hipStream_t stream);

}  // namespace kf
