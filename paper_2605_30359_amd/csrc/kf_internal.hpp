// Internal types shared by the host planner and the kernels of libkf.so.
#pragma once

#include <stdint.h>

#include "kf.h"

namespace kf {

struct EpiOp {
  int32_t kind;
  int32_t groups;
  float p0;
  float p1;
};

struct EpiProgram {
  int32_t n;
  EpiOp op[KF_MAX_OPS];
};

// A row op: one whose reduction runs over a whole row (the last op).
constexpr bool is_row_op(int kind) {
  return kind == KF_OP_ROW_SOFTMAX || kind == KF_OP_ROW_LOGSUMEXP || kind == KF_OP_ROW_CROSS_ENTROPY;
}
// Compile-time shape of an epilogue: element-wise ops only, or element-wise
// ops around one GroupNorm, or element-wise ops followed by a row softmax /
// logsumexp.
enum EpiShape { kEpiPlain = 0, kEpiGroupNorm = 1, kEpiRow = 2 };

// Op chains with an epilogue generated for exactly that op sequence (the op
// parameters stay run-time values).  Chain 0 is the general one: the op list
// is interpreted at run time.  The paper turns each operator into its own
// specialised kernel; these are the chains of the benchmarked operators and
// the plain building blocks, and every other chain runs interpreted.
constexpr int kNumChains = 15;
constexpr int kChainLen[kNumChains] = {0, 0, 1, 2, 4, 3, 3, 3, 5, 1, 4, 1, 1, 1, 2};
constexpr int kChainOps[kNumChains][KF_MAX_OPS] = {
    {},                                                                         // 0: interpreted
    {},                                                                         // 1: contraction only
    {KF_OP_BIAS},                                                               // 2
    {KF_OP_BIAS, KF_OP_RELU},                                                   // 3
    {KF_OP_BIAS, KF_OP_GELU_TANH, KF_OP_SCALE, KF_OP_ROW_LOGSUMEXP},           // 4: GEMM, GELU, logsumexp
    {KF_OP_GROUPNORM, KF_OP_SWISH, KF_OP_RESIDUAL_ADD},                        // 5: GEMM, GroupNorm, swish
    {KF_OP_BIAS, KF_OP_HARDTANH, KF_OP_ROW_SOFTMAX},                           // 6: GEMM, hardtanh, softmax
    {KF_OP_BIAS, KF_OP_RELU, KF_OP_MAXPOOL2X2},                                // 7: conv, ReLU, max-pool
    {KF_OP_BIAS, KF_OP_SWISH, KF_OP_TANH, KF_OP_GELU_ERF, KF_OP_HARDTANH},     // 8: GEMM + activation chain
    {KF_OP_ROW_SOFTMAX},                                                        // 9: softmax rows
    {KF_OP_BIAS, KF_OP_CHANNEL_SOFTMAX, KF_OP_MAXPOOL3D_2, KF_OP_MAXPOOL3D_2},  // 10: conv3d, softmax, pools
    {KF_OP_GROUPNORM},                                                          // 11: GroupNorm rows
    {KF_OP_ROW_LOGSUMEXP},                                                      // 12: logsumexp rows
    {KF_OP_ROW_CROSS_ENTROPY},                                                  // 13: cross-entropy rows
    {KF_OP_BIAS, KF_OP_ROW_CROSS_ENTROPY},                                      // 14: GEMM + bias, cross-entropy
};
// Which contraction a chain belongs to: 0 any, 1 GEMM / ROWWISE, 2 CONV2D_3X3,
// 3 CONV3D_3X3X3.
constexpr int kChainFamily[kNumChains] = {0, 0, 1, 1, 1, 1, 1, 2, 1, 1, 3, 1, 1, 1, 1};
// Chains of one row reduction (the unfused comparator's row-op kernels).
constexpr int kChainRowSoftmax = 9;
constexpr int kChainGroupNorm = 11;
constexpr int kChainRowLogsumexp = 12;
constexpr int kChainRowCrossEntropy = 13;

// Arguments of the GEMM-shaped kernels (passed by value as kernel arguments).
struct GemmArgs {
  const void* a;          // [M, lda] row-major
  const void* b;          // [K, ldb] (KN) or [N, ldb] (NK)
  int64_t M, N, K;
  int64_t lda, ldb;
  EpiProgram prog;
  const float* bias;      // [N] or null
  const float* gamma;     // [N] or null
  const float* beta;      // [N] or null
  const void* residual;   // [M, ldr] or null
  int64_t ldr;
  int32_t residual_bf16;
  int32_t out_bf16;
  void* out;              // [M, ldo] (or [M] for a row logsumexp)
  int64_t ldo;
  void* partials;         // float2 [M][tiles_n] for row softmax / logsumexp / cross-entropy
  const int32_t* targets; // [M] class targets (ROW_CROSS_ENTROPY) or null
  float* tlogit;          // [M] h[m][target_m], written by the tile holding it
  int32_t tiles_m, tiles_n;
  int32_t gn_group;       // GroupNorm group width in columns (0 = none)
  int32_t red_index;      // position of the reduction op in prog (n if none)
  float scale;            // dequantisation factor applied to the accumulator
  int32_t raster_group;   // tile rows walked together (column by column) by consecutive tiles
  int32_t xcd_remap;      // 1: each XCD takes a contiguous range of tiles
  int32_t stage_out;      // 256x256 kernel: 1 = bf16 output row blocks go through LDS (coalesced stores)
  long long* stamps;      // 256x256 kernel: 4 counters per workgroup (see kf_set_clock_stamps) or null
  int64_t stamp_cap;      // workgroups stamps has room for
};

// Arguments of the row-wise kernel (no contraction: h = A).
struct RowArgs {
  const void* a;          // [M, lda]
  int64_t M, N, lda;
  int32_t in_bf16;
  EpiProgram prog;
  const float* bias;      // [N] or null
  const float* gamma;     // [N] or null
  const float* beta;      // [N] or null
  const void* residual;   // [M, ldr] or null
  int64_t ldr;
  int32_t residual_bf16;
  int32_t out_bf16;
  void* out;              // [M, ldo] (or [M] for a row logsumexp / cross-entropy)
  int64_t ldo;
  int32_t gn_group;       // GroupNorm group width in columns (0 = none)
  const int32_t* targets; // [M] class targets (ROW_CROSS_ENTROPY) or null
};

// Arguments of the implicit-GEMM 3x3 convolution kernels.
struct ConvArgs {
  const void* x;          // [batch, cin, H, W]
  const void* w;          // [cout, cin, 3, 3]
  int64_t batch, cin, H, W, cout;
  EpiProgram prog;
  const float* bias;      // [cout] or null
  const void* residual;   // output-shaped or null
  int32_t residual_bf16;
  int32_t out_bf16;
  void* out;              // [batch, cout, H(/2), W(/2)]
  int32_t pool;           // 1 if the op list ends with a 2x2 max-pool
  int32_t pool_index;     // position of the pool op in prog
  int32_t tiles;          // number of output tiles (batch x H/2 row pairs)
  int32_t grid;           // workgroups of the persistent launch (at most tiles)
  int32_t variant;        // 0: 4 waves (128 x 64 wave blocks), 1: 8 waves (64 x 64), 2: general shapes
};

// Arguments of the implicit-GEMM 3x3x3 convolution kernel.
struct Conv3dArgs {
  const void* x;          // [batch][D][H][W][cin] (channels-last)
  int32_t batch, D, H, W;
  EpiProgram prog;
  const float* bias;      // [cout] or null
  void* out;              // [batch, cout, Dp, Hp, Wp] (NCDHW)
  int32_t pools;          // 0, or 2 (two MaxPool3d(2) = max over 4x4x4 blocks)
  int32_t Dp, Hp, Wp;     // output extents (after the pools)
  int32_t tiles_d, tiles_h, tiles_w;  // output tiles of 4 x 4 x 16 conv positions
  int32_t tiles;          // batch * tiles_d * tiles_h * tiles_w
  int32_t grid;           // workgroups of the persistent launch
  int32_t xcd_remap;      // 1: the workgroups of one XCD take consecutive tiles
};

}  // namespace kf
