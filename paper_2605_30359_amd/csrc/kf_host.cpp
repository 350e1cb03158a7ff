// libkf.so host side: the C ABI declared in include/kf.h.
//
// kf_create validates an op descriptor on the host (no device call), then
// checks for a gfx950 device and allocates the descriptor's workspace.
// kf_fused_op checks the caller's tensors against the plan and enqueues the
// kernels on the caller's stream.  Nothing here throws or aborts across the
// ABI; every failure is a status code plus a thread-local message.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "kf.h"
#include "kf_internal.hpp"
#include "kf_launch.hpp"

namespace {

// The message of the last failing call on this thread: a fixed buffer, so
// that reporting an error allocates nothing.
thread_local char g_last_error[512];

kf_status fail(kf_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

kf_status ok() {
  g_last_error[0] = '\0';
  return KF_OK;
}

enum Variant { kVarGemmF32 = 0, kVarGemmBf16 = 1, kVarGemmFp8 = 2, kVarConvBf16 = 3, kVarRowwise = 4, kVarConv3d = 5 };

struct Slot {
  int32_t dtype;
  int32_t ndim;
  int64_t shape[KF_MAX_DIMS];
  const char* name;
  bool channels_last;  // a 5-D [N, C, D, H, W] tensor stored as [N][D][H][W][C]
  bool or_dense = false;  // channels_last slot that also takes a contiguous [N, C, D, H, W]
};

// The input slots of a plan: A, B and at most one bias, gamma, beta and
// residual -- a fixed-capacity list, so that a plan can live on the stack.
constexpr int kMaxSlots = 6;
struct SlotList {
  Slot s[kMaxSlots];
  int n = 0;
  void clear() { n = 0; }
  void push_back(const Slot& x) {
    if (n < kMaxSlots) s[n++] = x;
  }
  size_t size() const { return (size_t)n; }
  const Slot& operator[](size_t i) const { return s[i]; }
  const Slot* begin() const { return s; }
  const Slot* end() const { return s + n; }
};

// Rows a one-workgroup-per-row launch (256 threads each) can cover.
constexpr int64_t kMaxRowLaunch = int64_t(1) << 24;

int64_t elem_size(int32_t dt) { return dt == KF_F32 || dt == KF_I32 ? 4 : dt == KF_BF16 ? 2 : 1; }

bool is_elementwise_kind(int k) {
  return k == KF_OP_RELU || k == KF_OP_GELU_TANH || k == KF_OP_GELU_ERF || k == KF_OP_SWISH ||
         k == KF_OP_SIGMOID || k == KF_OP_TANH || k == KF_OP_HARDTANH || k == KF_OP_SCALE;
}

}  // namespace

struct kf_desc {
  int num_cu = 1;  // compute units of the device (persistent launch width)
  kf_op_spec spec;
  Variant variant;
  kf::EpiProgram prog;
  int epi_shape;
  int red_index;
  int gn_group;
  int row_kind;  // KF_OP_ROW_SOFTMAX / KF_OP_ROW_LOGSUMEXP / KF_OP_ROW_CROSS_ENTROPY / 0
  int chain = 0;  // compile-time epilogue chain matching the op list (0: interpreted)
  bool conv_special = false;  // CONV2D_3X3 in the tiled kernels' shape family
  bool conv3d_tiled = false;  // CONV3D_3X3X3 in the tiled kernel's shape family (cin 16, cout 64)
  int conv3d_split = 0;       // CONV3D_3X3X3: ops [0, split) are BIAS / element-wise (the general kernel fuses them)
  SlotList inputs;
  Slot output;
  int device;
  void* workspace;
  size_t workspace_bytes;
  int tiles_n;
  const char* kernel_name = "";
  kf_tuning tuning;  // launch fields (see kf_set_tuning)
  // unfused comparator: two intermediate buffers, allocated on first use
  mutable void* ubuf[2];
  mutable size_t ubuf_bytes;
  // conv plans: the weight tensor whose repacked copy the workspace holds
  // (nullptr: none yet, or the caller declared the weights changed)
  mutable const void* packed_from = nullptr;
  mutable int packed_kind = 0;  // conv3d: 1 = packed for the tiled kernel, 2 = for the general one
  // GEMM: the caller's buffer for per-workgroup clock stamps (or null)
  long long* stamps = nullptr;
  int64_t stamp_cap = 0;
};

namespace {

// The compile-time chain whose op kinds equal the spec's and which belongs to
// the spec's contraction (chain 1, no ops, to every one), else 0.  A GEMM
// chain whose row reduction follows a HARDTANH is compiled for that
// HARDTANH's upper bound as the row offset, valid for bounds at most 64
// apart; with wider bounds the op runs interpreted.
int match_chain(const kf_op_spec* s) {
  const int family = s->contraction == KF_CONV2D_3X3 ? 2 : s->contraction == KF_CONV3D_3X3X3 ? 3 : 1;
  for (int ch = 1; ch < kf::kNumChains; ++ch) {
    if ((kf::kChainFamily[ch] != 0 && kf::kChainFamily[ch] != family) || kf::kChainLen[ch] != s->n_ops) continue;
    bool same = true;
    for (int o = 0; o < s->n_ops; ++o) same = same && s->ops[o].kind == kf::kChainOps[ch][o];
    if (!same) continue;
    if (s->contraction == KF_GEMM)
      for (int o = 1; o < s->n_ops; ++o)
        if (kf::is_row_op(s->ops[o].kind) && s->ops[o - 1].kind == KF_OP_HARDTANH &&
            !(s->ops[o - 1].p1 - s->ops[o - 1].p0 <= 64.0f))
          return 0;
    return ch;
  }
  return 0;
}

kf_status validate_and_plan(const kf_op_spec* s, kf_desc* d) {
  if (!s) return fail(KF_ERR_INVALID_ARG, "spec is NULL");
  if (s->contraction != KF_GEMM && s->contraction != KF_CONV2D_3X3 && s->contraction != KF_ROWWISE &&
      s->contraction != KF_CONV3D_3X3X3)
    return fail(KF_ERR_INVALID_ARG, "unknown contraction %d", s->contraction);
  if (s->in_dtype != KF_F32 && s->in_dtype != KF_BF16 && s->in_dtype != KF_FP8_E4M3)
    return fail(KF_ERR_INVALID_ARG, "unknown in_dtype %d", s->in_dtype);
  if (s->out_dtype != KF_F32 && s->out_dtype != KF_BF16)
    return fail(KF_ERR_INVALID_ARG, "out_dtype must be KF_F32 or KF_BF16 (got %d)", s->out_dtype);
  if (s->n_ops < 0 || s->n_ops > KF_MAX_OPS)
    return fail(KF_ERR_INVALID_ARG, "n_ops must be in [0, %d] (got %d)", KF_MAX_OPS, s->n_ops);

  memset(&d->prog, 0, sizeof(d->prog));
  d->prog.n = s->n_ops;
  d->red_index = s->n_ops;
  d->epi_shape = kf::kEpiPlain;
  d->gn_group = 0;
  d->row_kind = 0;
  int n_red = 0, n_pool = 0, n_pool3 = 0, n_csm = 0;
  bool has_bias = false, has_gn = false, has_res = false;
  for (int i = 0; i < s->n_ops; ++i) {
    const kf_op& op = s->ops[i];
    if (op.kind < KF_OP_BIAS || op.kind > KF_OP_ROW_CROSS_ENTROPY)
      return fail(KF_ERR_INVALID_ARG, "op %d: unknown kind %d", i, op.kind);
    d->prog.op[i] = kf::EpiOp{op.kind, op.groups, op.p0, op.p1};
    switch (op.kind) {
      case KF_OP_BIAS:
        if (has_bias) return fail(KF_ERR_UNSUPPORTED, "op %d: at most one BIAS op", i);
        has_bias = true;
        break;
      case KF_OP_HARDTANH:
        if (!(op.p0 <= op.p1)) return fail(KF_ERR_INVALID_ARG, "op %d: HARDTANH needs lo <= hi", i);
        break;
      case KF_OP_GROUPNORM:
        if (has_gn) return fail(KF_ERR_UNSUPPORTED, "op %d: at most one GROUPNORM op", i);
        has_gn = true;
        if (op.groups < 1) return fail(KF_ERR_INVALID_ARG, "op %d: GROUPNORM groups must be >= 1", i);
        if (!(op.p0 >= 0.0f) || !std::isfinite(op.p0))
          return fail(KF_ERR_INVALID_ARG, "op %d: GROUPNORM eps must be finite and >= 0", i);
        ++n_red;
        d->red_index = i;
        d->epi_shape = kf::kEpiGroupNorm;
        break;
      case KF_OP_RESIDUAL_ADD:
        if (has_res) return fail(KF_ERR_UNSUPPORTED, "op %d: at most one RESIDUAL_ADD op", i);
        has_res = true;
        if (s->residual_dtype != KF_F32 && s->residual_dtype != KF_BF16)
          return fail(KF_ERR_INVALID_ARG, "residual_dtype must be KF_F32 or KF_BF16");
        break;
      case KF_OP_MAXPOOL2X2:
        ++n_pool;
        if (s->contraction != KF_CONV2D_3X3) return fail(KF_ERR_UNSUPPORTED, "op %d: MAXPOOL2X2 needs CONV2D_3X3", i);
        break;
      case KF_OP_ROW_SOFTMAX:
      case KF_OP_ROW_LOGSUMEXP:
      case KF_OP_ROW_CROSS_ENTROPY:
        if (i != s->n_ops - 1) return fail(KF_ERR_UNSUPPORTED, "op %d: a row softmax/logsumexp must be the last op", i);
        if (s->contraction != KF_GEMM && s->contraction != KF_ROWWISE)
          return fail(KF_ERR_UNSUPPORTED, "op %d: row ops need a GEMM or ROWWISE", i);
        ++n_red;
        d->red_index = i;
        d->epi_shape = kf::kEpiRow;
        d->row_kind = op.kind;
        break;
      case KF_OP_CHANNEL_SOFTMAX:
        if (s->contraction != KF_CONV3D_3X3X3)
          return fail(KF_ERR_UNSUPPORTED, "op %d: CHANNEL_SOFTMAX needs CONV3D_3X3X3", i);
        if (n_pool3) return fail(KF_ERR_UNSUPPORTED, "op %d: CHANNEL_SOFTMAX must come before the pools", i);
        ++n_csm;
        break;
      case KF_OP_MAXPOOL3D_2:
        if (s->contraction != KF_CONV3D_3X3X3)
          return fail(KF_ERR_UNSUPPORTED, "op %d: MAXPOOL3D_2 needs CONV3D_3X3X3", i);
        ++n_pool3;
        break;
      default:
        break;
    }
    if (n_pool3 && op.kind != KF_OP_MAXPOOL3D_2)
      return fail(KF_ERR_UNSUPPORTED, "op %d: the MAXPOOL3D_2 ops must be the last ops", i);
  }
  if (n_csm > 1) return fail(KF_ERR_UNSUPPORTED, "at most one CHANNEL_SOFTMAX op");
  if (n_red > 1) return fail(KF_ERR_UNSUPPORTED, "at most one reduction op (GROUPNORM / ROW_*) per chain");
  if (n_pool > 1) return fail(KF_ERR_UNSUPPORTED, "at most one MAXPOOL2X2 op");
  const bool row_scalar = d->row_kind == KF_OP_ROW_LOGSUMEXP || d->row_kind == KF_OP_ROW_CROSS_ENTROPY;
  if (row_scalar && s->out_dtype != KF_F32)
    return fail(KF_ERR_UNSUPPORTED, "ROW_LOGSUMEXP / ROW_CROSS_ENTROPY output must be KF_F32");
  // the row kernels (row softmax / logsumexp finish, the row-wise chains)
  // launch one 256-thread workgroup per row, and a launch holds fewer than
  // 2^32 work-items
  if ((d->row_kind || s->contraction == KF_ROWWISE) && s->M >= kMaxRowLaunch)
    return fail(KF_ERR_UNSUPPORTED, "row reductions support M < %lld rows (one workgroup per row)",
                (long long)kMaxRowLaunch);

  const int32_t dt = s->in_dtype;
  d->inputs.clear();
  if (s->contraction == KF_GEMM) {
    if (s->M < 0 || s->N < 1 || s->K < 0) return fail(KF_ERR_SHAPE, "GEMM needs M >= 0, N >= 1, K >= 0");
    if (s->M > INT32_MAX || s->N > INT32_MAX || s->K > INT32_MAX) return fail(KF_ERR_UNSUPPORTED, "GEMM sizes must be < 2^31");
    if (s->b_layout != KF_LAYOUT_KN && s->b_layout != KF_LAYOUT_NK) return fail(KF_ERR_INVALID_ARG, "unknown b_layout %d", s->b_layout);
    const bool nk = s->b_layout == KF_LAYOUT_NK;
    d->inputs.push_back(Slot{dt, 2, {s->M, s->K, 0, 0, 0}, "A", false});
    d->inputs.push_back(Slot{dt, 2, {nk ? s->N : s->K, nk ? s->K : s->N, 0, 0, 0}, "B", false});
    if (dt == KF_F32) {
      d->variant = kVarGemmF32;
      if (d->epi_shape != kf::kEpiPlain)
        return fail(KF_ERR_UNSUPPORTED, "fp32 GEMM supports element-wise, BIAS and RESIDUAL_ADD ops only");
      if ((s->M + 7) / 8 > 65535) return fail(KF_ERR_UNSUPPORTED, "fp32 GEMM supports M <= 524280");
      d->kernel_name = "kf_gemm_f32_8x8";
    } else if (dt == KF_BF16) {
      d->variant = kVarGemmBf16;
      if (s->K % 8) return fail(KF_ERR_UNSUPPORTED, "bf16 GEMM needs K %% 8 == 0 (16-byte rows)");
      if (s->N % 8) return fail(KF_ERR_UNSUPPORTED, "bf16 GEMM needs N %% 8 == 0 (16-byte rows)");
      d->kernel_name = "kf_gemm_mfma_256x256";
    } else {
      d->variant = kVarGemmFp8;
      if (s->K % 16) return fail(KF_ERR_UNSUPPORTED, "fp8 GEMM needs K %% 16 == 0 (16-byte rows)");
      if (s->N % 16) return fail(KF_ERR_UNSUPPORTED, "fp8 GEMM needs N %% 16 == 0 (16-byte rows)");
      if (!(s->scale_a > 0.0f) || !(s->scale_b > 0.0f) || !std::isfinite(s->scale_a) || !std::isfinite(s->scale_b))
        return fail(KF_ERR_INVALID_ARG, "fp8 scale_a / scale_b must be finite and > 0");
      if (!std::isfinite(s->scale_a * s->scale_b) || s->scale_a * s->scale_b == 0.0f)
        return fail(KF_ERR_INVALID_ARG, "fp8 scale_a * scale_b must be a finite, nonzero fp32 value");
      d->kernel_name = "kf_gemm_mfma_256x256";
    }
    if (has_gn) {
      const kf_op& g = s->ops[d->red_index];
      if (s->N % g.groups) return fail(KF_ERR_SHAPE, "GROUPNORM: N=%lld not divisible by groups=%d", (long long)s->N, g.groups);
      d->gn_group = (int)(s->N / g.groups);
      if (d->gn_group != 128 && d->gn_group != 256)
        return fail(KF_ERR_UNSUPPORTED, "GROUPNORM: fused group width must be 128 or 256 columns (got %d)", d->gn_group);
    }
    for (int i = 0; i < s->n_ops; ++i) {
      const int k = s->ops[i].kind;
      if (k == KF_OP_BIAS) d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "bias", false});
      if (k == KF_OP_GROUPNORM) {
        d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "gamma", false});
        d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "beta", false});
      }
      if (k == KF_OP_RESIDUAL_ADD) d->inputs.push_back(Slot{s->residual_dtype, 2, {s->M, s->N, 0, 0, 0}, "residual", false});
    }
    if (d->row_kind == KF_OP_ROW_CROSS_ENTROPY)
      d->inputs.push_back(Slot{KF_I32, 1, {s->M, 0, 0, 0, 0}, "targets", false});
    if (row_scalar)
      d->output = Slot{KF_F32, 1, {s->M, 0, 0, 0, 0}, "out", false};
    else
      d->output = Slot{s->out_dtype, 2, {s->M, s->N, 0, 0, 0}, "out", false};
    if (d->row_kind) {
      d->tiles_n = (int)((s->N + kf::gemm_mfma_tile_n() - 1) / kf::gemm_mfma_tile_n());
      if (d->tiles_n > kf::row_finish_max_tiles())
        return fail(KF_ERR_UNSUPPORTED, "row softmax/logsumexp supports N <= %d", kf::row_finish_max_tiles() * kf::gemm_mfma_tile_n());
    }
  } else if (s->contraction == KF_ROWWISE) {
    // no contraction: the op list over the rows of A [M, N]
    if (dt != KF_F32 && dt != KF_BF16) return fail(KF_ERR_UNSUPPORTED, "ROWWISE supports fp32 and bf16 inputs");
    if (s->M < 0 || s->N < 1) return fail(KF_ERR_SHAPE, "ROWWISE needs M >= 0, N >= 1");
    if (s->M > INT32_MAX) return fail(KF_ERR_UNSUPPORTED, "ROWWISE supports M < 2^31");
    if (s->N % 8) return fail(KF_ERR_UNSUPPORTED, "ROWWISE needs N %% 8 == 0");
    if (kf::row_reduce_streams(d->prog) ? s->N > INT32_MAX : s->N > kf::rowwise_max_cols())
      return fail(KF_ERR_UNSUPPORTED,
                  "ROWWISE needs N <= %d (N < 2^31 for a row logsumexp / cross-entropy after element-wise ops)",
                  kf::rowwise_max_cols());
    if (has_gn) {
      const kf_op& g = s->ops[d->red_index];
      if (s->N % g.groups || (s->N / g.groups) % 8)
        return fail(KF_ERR_UNSUPPORTED, "GROUPNORM (ROWWISE): N / groups must be a whole multiple of 8 columns");
      d->gn_group = (int)(s->N / g.groups);
    }
    d->variant = kVarRowwise;
    d->kernel_name = kf::rowwise_kernel(d->prog, d->gn_group);
    d->inputs.push_back(Slot{dt, 2, {s->M, s->N, 0, 0, 0}, "A", false});
    for (int i = 0; i < s->n_ops; ++i) {
      const int k = s->ops[i].kind;
      if (k == KF_OP_BIAS) d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "bias", false});
      if (k == KF_OP_GROUPNORM) {
        d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "gamma", false});
        d->inputs.push_back(Slot{KF_F32, 1, {s->N, 0, 0, 0, 0}, "beta", false});
      }
      if (k == KF_OP_RESIDUAL_ADD) d->inputs.push_back(Slot{s->residual_dtype, 2, {s->M, s->N, 0, 0, 0}, "residual", false});
    }
    if (d->row_kind == KF_OP_ROW_CROSS_ENTROPY)
      d->inputs.push_back(Slot{KF_I32, 1, {s->M, 0, 0, 0, 0}, "targets", false});
    if (row_scalar)
      d->output = Slot{KF_F32, 1, {s->M, 0, 0, 0, 0}, "out", false};
    else
      d->output = Slot{s->out_dtype, 2, {s->M, s->N, 0, 0, 0}, "out", false};
  } else if (s->contraction == KF_CONV3D_3X3X3) {
    // 3x3x3 convolution, stride 1, no padding, channels-last input / OIDHW weight
    if (dt != KF_BF16) return fail(KF_ERR_UNSUPPORTED, "CONV3D_3X3X3 supports bf16 inputs only");
    if (s->out_dtype != KF_BF16) return fail(KF_ERR_UNSUPPORTED, "CONV3D_3X3X3 writes bf16 outputs only");
    if (s->batch < 0 || s->cin < 1 || s->cout < 1 || s->depth < 3 || s->height < 3 || s->width < 3)
      return fail(KF_ERR_SHAPE, "CONV3D_3X3X3 needs batch >= 0, cin, cout >= 1 and depth, height, width >= 3");
    // the tiled kernel: cin 16, cout 64, channels-last input, the whole op
    // family; every other shape or layout: the general kernel, BIAS and
    // element-wise ops
    d->conv3d_tiled = s->cin == kf::conv3d_cin() && s->cout == kf::conv3d_cout();
    // the general kernel fuses the leading BIAS / element-wise ops; a channel
    // softmax and the pools after them then run as one kernel each
    d->conv3d_split = 0;
    while (d->conv3d_split < s->n_ops && (s->ops[d->conv3d_split].kind == KF_OP_BIAS ||
                                          is_elementwise_kind(s->ops[d->conv3d_split].kind)))
      ++d->conv3d_split;
    if (d->conv3d_tiled && s->depth * s->height * s->width * s->cin * 2 >= (int64_t(1) << 30))
      return fail(KF_ERR_UNSUPPORTED, "one input volume must be smaller than 1 GiB");
    if (s->cin > (int64_t(1) << 20) || s->cout > (int64_t(1) << 20) ||
        kf::conv3d_gen_tiles(s->batch, s->depth, s->height, s->width, s->cout) > INT32_MAX)
      return fail(KF_ERR_UNSUPPORTED, "CONV3D_3X3X3 (general kernel) supports at most 2^31 - 1 tiles and 2^20 channels");
    if (n_pool3 != 0 && n_pool3 != 2)
      return fail(KF_ERR_UNSUPPORTED, "CONV3D_3X3X3 takes zero or two MAXPOOL3D_2 ops (got %d)", n_pool3);
    for (int i = 0; i < s->n_ops; ++i) {
      const int k = s->ops[i].kind;
      if (!(k == KF_OP_BIAS || k == KF_OP_CHANNEL_SOFTMAX || k == KF_OP_MAXPOOL3D_2 || is_elementwise_kind(k)))
        return fail(KF_ERR_UNSUPPORTED,
                    "op %d: CONV3D_3X3X3 supports BIAS, element-wise ops, CHANNEL_SOFTMAX and MAXPOOL3D_2", i);
    }
    int64_t od = s->depth - 2, oh = s->height - 2, ow = s->width - 2;
    // the unfused chain runs the conv alone over every position
    if (s->batch * ((od + 3) / 4) * ((oh + 3) / 4) * ((ow + 15) / 16) > INT32_MAX)
      return fail(KF_ERR_UNSUPPORTED, "CONV3D_3X3X3 supports at most 2^31 - 1 tiles");
    for (int i = 0; i < n_pool3; ++i) {
      od /= 2;
      oh /= 2;
      ow /= 2;
    }
    d->variant = kVarConv3d;
    d->kernel_name = d->conv3d_tiled ? "kf_conv3d_bf16_64x256" : "kf_conv3d_bf16_gen";
    // channels-last input; a contiguous NCDHW one too where the general
    // kernel can run the list
    d->inputs.push_back(Slot{dt, 5, {s->batch, s->cin, s->depth, s->height, s->width}, "A", true, true});
    d->inputs.push_back(Slot{dt, 5, {s->cout, s->cin, 3, 3, 3}, "B", false});
    for (int i = 0; i < s->n_ops; ++i)
      if (s->ops[i].kind == KF_OP_BIAS) d->inputs.push_back(Slot{KF_F32, 1, {s->cout, 0, 0, 0, 0}, "bias", false});
    d->output = Slot{KF_BF16, 5, {s->batch, s->cout, od, oh, ow}, "out", false};
  } else {
    // 3x3 convolution, stride 1, zero padding 1, NCHW input / OIHW weight
    if (dt != KF_BF16) return fail(KF_ERR_UNSUPPORTED, "CONV2D_3X3 supports bf16 inputs only");
    if (s->out_dtype != KF_BF16) return fail(KF_ERR_UNSUPPORTED, "CONV2D_3X3 writes bf16 outputs only");
    if (s->batch < 0 || s->cin < 1 || s->height < 1 || s->width < 1 || s->cout < 1)
      return fail(KF_ERR_SHAPE, "CONV2D_3X3 needs batch >= 0 and positive cin, height, width, cout");
    if (n_pool && (s->height % 2 || s->width % 2))
      return fail(KF_ERR_UNSUPPORTED, "MAXPOOL2X2 needs an even height and width");
    if ((int64_t)std::max(s->cin, s->cout) * s->height * s->width * 2 >= (int64_t(1) << 31) || s->cin > (1 << 20) ||
        s->cout > (1 << 20))
      return fail(KF_ERR_UNSUPPORTED, "one input or output image must be smaller than 2 GiB");
    // the tiled kernels are built for the 64 -> 128 channel, 128-column family
    // with even height; every other shape takes the general kernel
    d->conv_special = s->cin == kf::conv_bf16_cin() && s->width == kf::conv_bf16_width() &&
                      s->cout == kf::conv_bf16_cout() && s->height % 2 == 0;
    if (d->conv_special && (int64_t)s->batch * (s->height / 2) > INT32_MAX)
      return fail(KF_ERR_UNSUPPORTED, "CONV2D_3X3 supports at most 2^31 - 1 row-pair tiles");
    if (!d->conv_special && kf::conv_gen_tiles(s->batch, s->height, s->width, s->cout) >= (int64_t(1) << 24))
      return fail(KF_ERR_UNSUPPORTED, "CONV2D_3X3 (general shapes) supports fewer than 2^24 tiles of 4 x 32 x 128");
    for (int i = 0; i < s->n_ops; ++i) {
      const int k = s->ops[i].kind;
      if (!(k == KF_OP_BIAS || k == KF_OP_MAXPOOL2X2 || is_elementwise_kind(k)))
        return fail(KF_ERR_UNSUPPORTED, "op %d: CONV2D_3X3 supports BIAS, element-wise ops and MAXPOOL2X2", i);
    }
    d->variant = kVarConvBf16;
    d->kernel_name = d->conv_special ? "kf_conv3x3_bf16_256x128" : "kf_conv3x3_bf16_gen";
    // the 8-wave tile is the faster at the C4 shape (the tuner may pick any)
    d->tuning.variant = d->conv_special ? 1 : 2;
    d->inputs.push_back(Slot{dt, 4, {s->batch, s->cin, s->height, s->width}, "A", false});
    d->inputs.push_back(Slot{dt, 4, {s->cout, s->cin, 3, 3}, "B", false});
    for (int i = 0; i < s->n_ops; ++i)
      if (s->ops[i].kind == KF_OP_BIAS) d->inputs.push_back(Slot{KF_F32, 1, {s->cout, 0, 0, 0, 0}, "bias", false});
    if (n_pool)
      d->output = Slot{KF_BF16, 4, {s->batch, s->cout, s->height / 2, s->width / 2}, "out", false};
    else
      d->output = Slot{KF_BF16, 4, {s->batch, s->cout, s->height, s->width}, "out", false};
  }
  return KF_OK;
}

kf_status check_tensor(const kf_tensor* t, const Slot& s, bool is_output, bool vec16) {
  const char* what = is_output ? "output" : "input";
  if (t->dtype != s.dtype) return fail(KF_ERR_SHAPE, "%s '%s': dtype %d, expected %d", what, s.name, t->dtype, s.dtype);
  if (t->ndim != s.ndim) return fail(KF_ERR_SHAPE, "%s '%s': ndim %d, expected %d", what, s.name, t->ndim, s.ndim);
  int64_t numel = 1;
  for (int i = 0; i < s.ndim; ++i) {
    if (t->shape[i] != s.shape[i])
      return fail(KF_ERR_SHAPE, "%s '%s': shape[%d] = %lld, expected %lld", what, s.name, i, (long long)t->shape[i], (long long)s.shape[i]);
    numel *= s.shape[i];
  }
  if (numel == 0) return KF_OK;  // never dereferenced
  if (!t->data) return fail(KF_ERR_INVALID_ARG, "%s '%s': data is NULL", what, s.name);
  if (s.channels_last) {
    // [N, C, D, H, W] with strides [D H W C, 1, H W C, W C, C]
    const int64_t C = s.shape[1];
    const int64_t expect[5] = {s.shape[2] * s.shape[3] * s.shape[4] * C, 1, s.shape[3] * s.shape[4] * C,
                               s.shape[4] * C, C};
    bool cl = true, dense = s.or_dense;
    int64_t run = 1;
    for (int i = 4; i >= 0; --i) {
      if (t->stride[i] != expect[i] && s.shape[i] != 1) cl = false;
      if (t->stride[i] != run && s.shape[i] != 1) dense = false;
      run *= s.shape[i];
    }
    if (!cl && !dense)
      return fail(KF_ERR_UNSUPPORTED, "%s '%s': must be channels-last (torch.channels_last_3d)%s and dense", what,
                  s.name, s.or_dense ? " or contiguous NCDHW" : "");
  } else if (t->stride[s.ndim - 1] != 1) {
    return fail(KF_ERR_UNSUPPORTED, "%s '%s': innermost stride must be 1", what, s.name);
  }
  const int64_t es = elem_size(s.dtype);
  const int64_t align = vec16 ? 16 : es;
  if (reinterpret_cast<uintptr_t>(t->data) % align)
    return fail(KF_ERR_UNSUPPORTED, "%s '%s': data must be %lld-byte aligned", what, s.name, (long long)align);
  if (s.ndim == 2) {
    if (t->stride[0] < s.shape[1]) return fail(KF_ERR_SHAPE, "%s '%s': row stride %lld < row length %lld", what, s.name, (long long)t->stride[0], (long long)s.shape[1]);
    if (vec16 && (t->stride[0] * es) % 16)
      return fail(KF_ERR_UNSUPPORTED, "%s '%s': row stride must be a multiple of 16 bytes", what, s.name);
  } else if (s.ndim >= 4 && !s.channels_last) {
    int64_t expect = 1;
    for (int i = s.ndim - 1; i >= 0; --i) {
      if (t->stride[i] != expect && s.shape[i] != 1)
        return fail(KF_ERR_UNSUPPORTED, "%s '%s': %d-D tensors must be contiguous", what, s.name, s.ndim);
      expect *= s.shape[i];
    }
  }
  return KF_OK;
}

// Byte extents addressed through 32-bit buffer offsets must stay below 2^31.
bool fits_31(int64_t bytes) { return bytes >= 0 && bytes < (int64_t(1) << 31); }

// Kernel arguments of a CONV3D_3X3X3 plan; pools = 0 stores every conv
// output position, pools = 2 the 4x4x4-block maxima.  inputs may be NULL
// (the launch shape alone, for planning): then no tensor pointer is set.
kf::Conv3dArgs conv3d_args(const kf_desc* d, const kf_tensor* inputs, void* out, int pools) {
  const kf_op_spec& s = d->spec;
  kf::Conv3dArgs a;
  memset(&a, 0, sizeof(a));
  a.batch = (int32_t)s.batch;
  a.D = (int32_t)s.depth;
  a.H = (int32_t)s.height;
  a.W = (int32_t)s.width;
  a.prog = d->prog;
  if (inputs) {
    a.x = inputs[0].data;
    for (int i = 0; i < s.n_ops; ++i)
      if (s.ops[i].kind == KF_OP_BIAS) a.bias = static_cast<const float*>(inputs[2].data);
  }
  a.out = out;
  a.pools = pools;
  const int64_t od = s.depth - 2, oh = s.height - 2, ow = s.width - 2;
  a.Dp = (int32_t)(pools ? od / 4 : od);
  a.Hp = (int32_t)(pools ? oh / 4 : oh);
  a.Wp = (int32_t)(pools ? ow / 4 : ow);
  // conv positions the output needs, in tiles of 4 x 4 x 16
  const int64_t nd = pools ? 4 * (int64_t)a.Dp : od, nh = pools ? 4 * (int64_t)a.Hp : oh,
                nw = pools ? 4 * (int64_t)a.Wp : ow;
  a.tiles_d = (int32_t)((nd + 3) / 4);
  a.tiles_h = (int32_t)((nh + 3) / 4);
  a.tiles_w = (int32_t)((nw + 15) / 16);
  a.tiles = (int32_t)(s.batch * a.tiles_d * a.tiles_h * a.tiles_w);
  a.grid = d->tuning.wg_per_cu * d->num_cu;  // persistent: wg_per_cu workgroups per compute unit
  a.xcd_remap = d->tuning.xcd_remap;
  return a;
}

int conv3d_pool_count(const kf_op_spec& s) {
  int n = 0;
  for (int i = 0; i < s.n_ops; ++i) n += s.ops[i].kind == KF_OP_MAXPOOL3D_2;
  return n;
}

// The tiled conv3d kernel takes this call: a plan in its shape family with a
// channels-last input (channel stride 1; a contiguous NCDHW input has a
// channel stride of D H W >= 27).
bool conv3d_uses_tiled(const kf_desc* d, const kf_tensor* inputs) {
  return d->conv3d_tiled && inputs[0].stride[1] == 1;
}

// Kernel arguments of the general conv3d kernel (op list `prog`: the plan's,
// or none for the unfused chain's convolution).
kf::Conv3dGenArgs conv3d_gen_args(const kf_desc* d, const kf_tensor* inputs, void* out, const kf::EpiProgram& prog) {
  const kf_op_spec& s = d->spec;
  kf::Conv3dGenArgs g;
  memset(&g, 0, sizeof(g));
  const kf_tensor& x = inputs[0];
  g.x = x.data;
  g.sn = x.stride[0];
  g.sc = x.stride[1];
  g.sd = x.stride[2];
  g.sh = x.stride[3];
  g.sw = x.stride[4];
  g.batch = (int32_t)s.batch;
  g.cin = (int32_t)s.cin;
  g.cout = (int32_t)s.cout;
  g.D = (int32_t)s.depth;
  g.H = (int32_t)s.height;
  g.W = (int32_t)s.width;
  g.prog = prog;
  for (int i = 0; i < prog.n; ++i)
    if (prog.op[i].kind == KF_OP_BIAS) g.bias = static_cast<const float*>(inputs[2].data);
  g.out = out;
  return g;
}

// Repack a conv3d plan's weights into ws for the kernel this call takes,
// unless ws already holds them (keep: the descriptor's own workspace).
hipError_t conv3d_pack(const kf_desc* d, void* ws, bool keep, bool tiled, const void* w, hipStream_t hs) {
  const int want = tiled ? 1 : 2;
  if (keep && d->packed_from == w && d->packed_kind == want) return hipSuccess;
  d->packed_from = nullptr;
  const hipError_t e = tiled ? kf::launch_conv3d_pack(w, ws, hs)
                             : kf::launch_conv3d_gen_pack(w, ws, (int)d->spec.cout, (int)d->spec.cin, hs);
  if (e == hipSuccess && keep) {
    d->packed_from = w;
    d->packed_kind = want;
  }
  return e;
}


// Algorithmic work of the plan's main kernel: FLOPs (2 per multiply-add of
// the contraction), bytes (each input read once, the output written once),
// workgroups launched and the dense peak of its arithmetic.
struct Work {
  double flops, bytes, peak_tflops;
  int64_t workgroups;
};

// Launch variant 1 of a GEMM plan: the 128x256 kernel, two persistent
// workgroups per CU (0: the 256x256 kernel).
int gemm_pp_workgroups(const kf_desc* d) {
  if ((d->variant != kVarGemmBf16 && d->variant != kVarGemmFp8) || d->tuning.variant != 1) return 0;
  const int64_t tiles = kf::gemm_pp_tiles(d->spec.M, d->spec.N);
  return (int)std::max<int64_t>(1, std::min<int64_t>(tiles, 2 * (int64_t)d->num_cu));
}

Work plan_work(const kf_desc* d) {
  const kf_op_spec& s = d->spec;
  Work w{0.0, 0.0, 157.3, 0};
  auto numel = [](const Slot& sl) {
    double n = 1.0;
    for (int i = 0; i < sl.ndim; ++i) n *= (double)sl.shape[i];
    return n;
  };
  for (const Slot& sl : d->inputs) w.bytes += numel(sl) * (double)elem_size(sl.dtype);
  w.bytes += numel(d->output) * (double)elem_size(d->output.dtype);
  switch (d->variant) {
    case kVarGemmF32:
      w.flops = 2.0 * s.M * s.N * s.K;
      w.workgroups = ((s.M + 7) / 8) * ((s.N + 7) / 8);
      break;
    case kVarGemmBf16:
    case kVarGemmFp8: {
      w.flops = 2.0 * s.M * s.N * s.K;
      w.peak_tflops = d->variant == kVarGemmFp8 ? 5033.2 : 2516.6;
      const int64_t bm = kf::gemm_mfma_tile_m(), bn = kf::gemm_mfma_tile_n();
      w.workgroups = d->tuning.variant == 1 ? gemm_pp_workgroups(d) : ((s.M + bm - 1) / bm) * ((s.N + bn - 1) / bn);
      break;
    }
    case kVarConvBf16:
      w.flops = 2.0 * s.batch * s.height * s.width * s.cout * s.cin * 9;
      w.peak_tflops = 2516.6;
      w.workgroups = d->tuning.variant == 2 ? kf::conv_gen_tiles(s.batch, s.height, s.width, s.cout)
                                            : std::min<int64_t>(d->num_cu, s.batch * (s.height / 2));
      break;
    case kVarConv3d: {
      w.flops = 2.0 * s.batch * (s.depth - 2) * (s.height - 2) * (s.width - 2) * s.cout * s.cin * 27;
      w.peak_tflops = 2516.6;
      int pools = 0;
      for (int i = 0; i < s.n_ops; ++i) pools += s.ops[i].kind == KF_OP_MAXPOOL3D_2;
      const kf::Conv3dArgs a = conv3d_args(d, nullptr, nullptr, pools);
      w.workgroups = d->conv3d_tiled ? std::min<int64_t>(a.grid, a.tiles)
                                     : kf::conv3d_gen_tiles(s.batch, s.depth, s.height, s.width, s.cout);
      break;
    }
    case kVarRowwise:
      w.workgroups = s.M;
      break;
  }
  return w;
}

void init_desc(kf_desc* d) {
  d->workspace = nullptr;
  d->workspace_bytes = 0;
  d->tiles_n = 0;
  d->ubuf[0] = d->ubuf[1] = nullptr;
  d->ubuf_bytes = 0;
  d->packed_from = nullptr;
  d->tuning = kf_tuning{4, 1, 2, 0};
}

// The current device, checked to be a gfx950, and its compute units; the
// properties are queried once per device and cached.
constexpr int kMaxDevices = 64;
std::atomic<int> g_device_cus[kMaxDevices];  // 0 unknown, -1 not gfx950, else the CU count

kf_status current_device(int* dev_out, int* cus_out) {
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count < 1) {
    (void)hipGetLastError();
    return fail(KF_ERR_NO_DEVICE, "no HIP device present");
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(KF_ERR_NO_DEVICE, "cannot query the current HIP device");
  }
  int cus = dev >= 0 && dev < kMaxDevices ? g_device_cus[dev].load(std::memory_order_relaxed) : 0;
  if (cus == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
      (void)hipGetLastError();
      return fail(KF_ERR_NO_DEVICE, "cannot query the current HIP device");
    }
    cus = strncmp(prop.gcnArchName, "gfx950", 6) != 0 ? -1 : (prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1);
    if (dev >= 0 && dev < kMaxDevices) g_device_cus[dev].store(cus, std::memory_order_relaxed);
    if (cus < 0) return fail(KF_ERR_NO_DEVICE, "device %d is %s; this library is built for gfx950 only", dev, prop.gcnArchName);
  }
  if (cus < 0) return fail(KF_ERR_NO_DEVICE, "device %d is not a gfx950; this library is built for gfx950 only", dev);
  *dev_out = dev;
  *cus_out = cus;
  return KF_OK;
}

// Device workspace a plan's kernels use: the repacked conv weights, or the
// per-(row, column tile) (max, sum) partials of a GEMM's row softmax /
// logsumexp.
size_t plan_workspace_bytes(const kf_desc* d) {
  const kf_op_spec& s = d->spec;
  if (d->variant == kVarConvBf16) return (size_t)9 * s.cout * kf::conv_gen_cin_pad((int)s.cin) * 2;
  if (d->variant == kVarConv3d) {
    const size_t gen = kf::conv3d_gen_packed_bytes(s.cout, s.cin);
    if (!d->conv3d_tiled) return gen;
    // the tiled kernel's packing, or the general one's for an NCDHW input
    return d->inputs.size() && d->inputs[0].or_dense ? std::max(kf::conv3d_packed_bytes(), gen)
                                                     : kf::conv3d_packed_bytes();
  }
  if (d->row_kind && d->variant != kVarRowwise) {
    // per-(row, tile) (max, sum) pairs; cross-entropy adds h[m][t_m] per row
    const size_t rows = (size_t)std::max<int64_t>(s.M, 1);
    return rows * d->tiles_n * sizeof(float) * 2 + (d->row_kind == KF_OP_ROW_CROSS_ENTROPY ? rows * sizeof(float) : 0);
  }
  return 0;
}

// Enqueue the fused operation of plan d with `ws` as its workspace.  The
// conv weights are repacked into ws unless `ws_keeps_weights` and ws already
// holds the repacked copy of this B tensor.
kf_status run_fused(const kf_desc* d, void* ws, bool ws_keeps_weights, const kf_tensor* inputs, kf_tensor* outputs,
                    void* stream, void* ev_before, void* ev_after);
kf_status run_chain_split(const kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream, int prefix,
                          void* ev_before, void* ev_after);

// latency-bound if the launch has fewer workgroups than compute units or
// reaches under 25% of both peaks, else the nearer roof (memory on a tie)
void classify_bound(kf_diagnosis* g) {
  constexpr double kLatencyFrac = 0.25;
  if (g->workgroups < g->compute_units || (g->compute_frac < kLatencyFrac && g->memory_frac < kLatencyFrac))
    g->bound = KF_BOUND_LATENCY;
  else
    g->bound = g->memory_frac >= g->compute_frac ? KF_BOUND_MEMORY : KF_BOUND_INSTRUCTION;
}

}  // namespace

extern "C" {

kf_status kf_probe_mfma(int32_t in_dtype, int64_t iters, kf_mfma_probe* out) {
  if (!out) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  memset(out, 0, sizeof(*out));
  if (in_dtype != KF_BF16 && in_dtype != KF_FP8_E4M3)
    return fail(KF_ERR_UNSUPPORTED, "the probe runs bf16 or fp8 e4m3 MFMAs");
  if (iters < 1 || iters > (int64_t(1) << 24)) return fail(KF_ERR_INVALID_ARG, "iters must be in [1, 2^24]");
  int dev = 0, cus = 0;
  kf_status st = current_device(&dev, &cus);
  if (st != KF_OK) return st;
  int wall_khz = 0;
  if (hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || wall_khz <= 0) {
    (void)hipGetLastError();
    return fail(KF_ERR_HIP, "cannot query the constant-rate counter's frequency");
  }
  const bool fp8 = in_dtype == KF_FP8_E4M3;
  const int wgs = cus;
  const size_t sink_bytes = (size_t)wgs * kf::probe_threads() * sizeof(float);
  const size_t stamp_bytes = (size_t)wgs * 4 * sizeof(long long);
  void* buf = nullptr;
  hipStream_t hs = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  std::vector<long long> stamps((size_t)wgs * 4);
  float ms = 0.0f;
  hipError_t e = hipMalloc(&buf, sink_bytes + stamp_bytes);
  if (e == hipSuccess) e = hipStreamCreate(&hs);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  float* sink = static_cast<float*>(buf);
  long long* st_dev = reinterpret_cast<long long*>(static_cast<char*>(buf) + sink_bytes);
  // an untimed launch of a tenth of the length first: clocks and power settle
  if (e == hipSuccess) e = kf::launch_mfma_probe(fp8, std::max<int64_t>(1, iters / 10), wgs, sink, st_dev, hs);
  if (e == hipSuccess) e = hipEventRecord(e0, hs);
  if (e == hipSuccess) e = kf::launch_mfma_probe(fp8, iters, wgs, sink, st_dev, hs);
  if (e == hipSuccess) e = hipEventRecord(e1, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess) e = hipMemcpy(stamps.data(), st_dev, stamp_bytes, hipMemcpyDeviceToHost);
  if (e != hipSuccess) (void)hipGetLastError();
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (hs) (void)hipStreamDestroy(hs);
  if (buf) (void)hipFree(buf);
  if (e != hipSuccess) return fail(KF_ERR_HIP, "probe failed: %s", hipGetErrorString(e));
  // shader clock of each workgroup: its clock ticks over its real time
  std::vector<double> ghz;
  for (int w = 0; w < wgs; ++w) {
    const long long dc = stamps[4 * w + 1] - stamps[4 * w], dw = stamps[4 * w + 3] - stamps[4 * w + 2];
    if (dc > 0 && dw > 0) ghz.push_back((double)dc / ((double)dw / ((double)wall_khz * 1e3)) * 1e-9);
  }
  std::sort(ghz.begin(), ghz.end());
  const double mfma_flops = fp8 ? 2.0 * 32 * 32 * 64 : 2.0 * 32 * 32 * 16;
  const double flops = (double)wgs * (kf::probe_threads() / 64) * (double)iters * 8 * mfma_flops;
  out->seconds = ms * 1e-3;
  out->tflops = ms > 0.0f ? flops / (ms * 1e-3) * 1e-12 : 0.0;
  out->clock_ghz = ghz.empty() ? 0.0 : ghz[ghz.size() / 2];
  out->workgroups = wgs;
  return ok();
}

kf_status kf_probe_copy(int64_t bytes, int32_t reps, kf_copy_probe* out) {
  if (!out) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  memset(out, 0, sizeof(*out));
  if (bytes < 16 || bytes % 16 || bytes > (int64_t(1) << 34))
    return fail(KF_ERR_INVALID_ARG, "bytes must be a multiple of 16 in [16, 2^34]");
  if (reps < 1 || reps > 1000) return fail(KF_ERR_INVALID_ARG, "reps must be in [1, 1000]");
  int dev = 0, cus = 0;
  kf_status st = current_device(&dev, &cus);
  if (st != KF_OK) return st;
  void* src = nullptr;
  void* dst = nullptr;
  hipStream_t hs = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float ms = 0.0f;
  const int64_t chunks = bytes / 16;
  hipError_t e = hipMalloc(&src, (size_t)bytes);
  if (e == hipSuccess) e = hipMalloc(&dst, (size_t)bytes);
  if (e == hipSuccess) e = hipStreamCreate(&hs);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  // one untimed copy (also fills the source), then `reps` timed back to back
  if (e == hipSuccess) e = hipMemsetAsync(src, 0x3c, (size_t)bytes, hs);
  if (e == hipSuccess) e = kf::launch_copy_probe(src, dst, chunks, hs);
  if (e == hipSuccess) e = hipEventRecord(e0, hs);
  for (int i = 0; i < reps && e == hipSuccess; ++i) e = kf::launch_copy_probe(src, dst, chunks, hs);
  if (e == hipSuccess) e = hipEventRecord(e1, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e != hipSuccess) (void)hipGetLastError();
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (hs) (void)hipStreamDestroy(hs);
  if (src) (void)hipFree(src);
  if (dst) (void)hipFree(dst);
  if (e != hipSuccess) {
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
      return fail(KF_ERR_OOM, "copy probe buffers of 2 x %lld bytes could not be allocated", (long long)bytes);
    return fail(KF_ERR_HIP, "probe failed: %s", hipGetErrorString(e));
  }
  out->seconds = ms * 1e-3 / reps;
  out->gbps = out->seconds > 0 ? 2.0 * (double)bytes / out->seconds * 1e-9 : 0.0;
  return ok();
}

kf_status kf_classify(double flops, double bytes, double seconds, double peak_tflops, double peak_gbps,
                      int64_t workgroups, int32_t compute_units, kf_diagnosis* out) {
  if (!out) return fail(KF_ERR_INVALID_ARG, "out is NULL");
  if (!(seconds > 0.0) || !(peak_tflops > 0.0) || !(peak_gbps > 0.0) || flops < 0.0 || bytes < 0.0)
    return fail(KF_ERR_INVALID_ARG, "seconds and peaks must be > 0, flops and bytes >= 0");
  kf_diagnosis& g = *out;
  g.flops = flops;
  g.bytes = bytes;
  g.seconds = seconds;
  g.tflops = flops / seconds * 1e-12;
  g.gbps = bytes / seconds * 1e-9;
  g.peak_tflops = peak_tflops;
  g.peak_gbps = peak_gbps;
  g.compute_frac = g.tflops / peak_tflops;
  g.memory_frac = g.gbps / peak_gbps;
  g.intensity = bytes > 0.0 ? flops / bytes : 0.0;
  g.ridge = peak_tflops * 1e12 / (peak_gbps * 1e9);
  g.workgroups = workgroups;
  g.compute_units = compute_units;
  g.mfma_busy = -1.0;
  g.lds_conflict = -1.0;
  g.traffic_ratio = -1.0;
  g.hints = 0;
  g.reserved = 0;
  classify_bound(&g);
  if (g.bound == KF_BOUND_LATENCY) g.hints |= workgroups < compute_units ? KF_HINT_PARALLELISM : KF_HINT_PIPELINE;
  return ok();
}

kf_status kf_diagnose(const kf_desc* d, double kernel_seconds, double hbm_bytes, kf_diagnosis* out) {
  if (!d || !out) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  const Work w = plan_work(d);
  return kf_classify(w.flops, hbm_bytes > 0.0 ? hbm_bytes : w.bytes, kernel_seconds, w.peak_tflops, 8000.0,
                     w.workgroups, d->num_cu, out);
}

kf_status kf_diagnose_counters(const kf_desc* d, const kf_counters* c, kf_diagnosis* out) {
  if (!d || !c || !out) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  const Work w = plan_work(d);
  const bool mfma = d->variant == kVarGemmBf16 || d->variant == kVarGemmFp8 || d->variant == kVarConvBf16 ||
                    d->variant == kVarConv3d;
  kf_status st = kf_classify(w.flops, c->hbm_bytes > 0.0 ? c->hbm_bytes : w.bytes, c->kernel_seconds, w.peak_tflops,
                             8000.0, w.workgroups, d->num_cu, out);
  if (st != KF_OK) return st;
  kf_diagnosis& g = *out;
  if (mfma && c->mfma_busy >= 0.0) {
    g.mfma_busy = c->mfma_busy;
    g.compute_frac = c->mfma_busy;  // the counted share of cycles the matrix cores worked
  }
  if (c->lds_conflict >= 0.0) g.lds_conflict = c->lds_conflict;
  if (c->hbm_bytes > 0.0 && w.bytes > 0.0) g.traffic_ratio = c->hbm_bytes / w.bytes;
  classify_bound(&g);
  g.hints = 0;
  if (g.workgroups < g.compute_units) g.hints |= KF_HINT_PARALLELISM;
  if (g.bound == KF_BOUND_LATENCY) g.hints |= KF_HINT_PIPELINE;
  if (g.traffic_ratio > 1.5 && (g.bound == KF_BOUND_MEMORY || mfma)) g.hints |= KF_HINT_REUSE;
  if (g.bound == KF_BOUND_INSTRUCTION && g.mfma_busy >= 0.0 && g.mfma_busy < 0.75) g.hints |= KF_HINT_OVERLAP;
  if (g.lds_conflict > 0.05) g.hints |= KF_HINT_LDS_LAYOUT;
  return ok();
}

kf_status kf_get_tuning(const kf_desc* d, kf_tuning* out) {
  if (!d || !out) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  *out = d->tuning;
  return ok();
}

kf_status kf_set_tuning(kf_desc* d, const kf_tuning* t) {
  if (!d || !t) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  if (t->raster_group < 1 || t->raster_group > 64) return fail(KF_ERR_INVALID_ARG, "raster_group must be in [1, 64]");
  if (t->xcd_remap != 0 && t->xcd_remap != 1) return fail(KF_ERR_INVALID_ARG, "xcd_remap must be 0 or 1");
  if (t->wg_per_cu != 1 && t->wg_per_cu != 2) return fail(KF_ERR_INVALID_ARG, "wg_per_cu must be 1 or 2");
  const bool gemm = d->variant == kVarGemmBf16 || d->variant == kVarGemmFp8;
  const int min_variant = d->variant == kVarConvBf16 && !d->conv_special ? 2 : 0;
  const int max_variant = d->variant == kVarConvBf16 || gemm ? 2 : 0;
  if (t->variant < min_variant || t->variant > max_variant)
    return fail(KF_ERR_INVALID_ARG, "variant must be in [%d, %d] for this plan", min_variant, max_variant);
  if (gemm && t->variant == 1 && d->spec.b_layout != KF_LAYOUT_KN)
    return fail(KF_ERR_INVALID_ARG, "variant 1 (128x256 tiles) takes B in KN layout only");
  d->tuning = *t;
  return ok();
}

namespace {

// Operand bytes the eight L2s fetch for a GEMM plan under launch
// configuration t (a model).  The grid has one workgroup per tile; workgroup
// b goes to XCD b % 8 and the device holds resident_per_cu x CUs of them at
// once, so consecutive ranges of that many workgroups run as rounds.  Within
// a round an XCD's L2 fetches each A panel (BM rows x K) and B panel (K x BN)
// that its tiles touch once; across rounds nothing is assumed to stay (a
// panel is 2-8 MiB against a 4 MiB L2).
double gemm_pp_panel_bytes(const kf_desc* d);

double gemm_panel_bytes(const kf_desc* d, const kf_tuning& t) {
  const kf_op_spec& s = d->spec;
  if (t.variant == 1) return gemm_pp_panel_bytes(d);
  const int64_t tm_n = (s.M + kf::gemm_mfma_tile_m() - 1) / kf::gemm_mfma_tile_m();
  const int64_t tn_n = (s.N + kf::gemm_mfma_tile_n() - 1) / kf::gemm_mfma_tile_n();
  const int64_t nwg = tm_n * tn_n;
  if (nwg <= 0 || nwg > (int64_t(1) << 22)) return -1.0;
  const double es = s.in_dtype == KF_FP8_E4M3 ? 1.0 : 2.0;
  const double a_panel = (double)kf::gemm_mfma_tile_m() * (double)s.K * es;
  const double b_panel = (double)kf::gemm_mfma_tile_n() * (double)s.K * es;
  const int64_t round = std::max<int64_t>(8, (int64_t)d->num_cu);  // one 256x256 workgroup per CU
  double bytes = 0.0;
  std::vector<uint8_t> seen_m((size_t)tm_n * 8), seen_n((size_t)tn_n * 8);
  for (int64_t r0 = 0; r0 < nwg; r0 += round) {
    std::fill(seen_m.begin(), seen_m.end(), 0);
    std::fill(seen_n.begin(), seen_n.end(), 0);
    for (int64_t bid = r0; bid < std::min(nwg, r0 + round); ++bid) {
      // the kernel's tile order (see tile_coords in the GEMM kernel)
      int64_t lid = bid;
      if (t.xcd_remap && (nwg & 7) == 0) lid = (bid & 7) * (nwg >> 3) + (bid >> 3);
      const int64_t per_group = (int64_t)t.raster_group * tn_n;
      const int64_t group = lid / per_group;
      const int64_t first_m = group * t.raster_group;
      const int64_t gsize = std::min<int64_t>(tm_n - first_m, t.raster_group);
      const int64_t rr = lid - group * per_group;
      const int64_t tm = first_m + rr % gsize, tn = rr / gsize;
      const int64_t x = bid & 7;
      uint8_t& fm = seen_m[(size_t)(tm * 8 + x)];
      uint8_t& fn = seen_n[(size_t)(tn * 8 + x)];
      if (!fm) bytes += a_panel;
      if (!fn) bytes += b_panel;
      fm = fn = 1;
    }
  }
  return bytes;
}

// The same model for the 128x256 kernel: G = 2 x CUs persistent workgroups,
// workgroup b on XCD b % 8 taking its i-th tile in round i, tiles ordered as
// the kernel orders them (each XCD a contiguous eighth, 8-row rasters).
double gemm_pp_panel_bytes(const kf_desc* d) {
  const kf_op_spec& s = d->spec;
  const int64_t tm_n = (s.M + 127) / 128;
  const int64_t tn_n = (s.N + kf::gemm_mfma_tile_n() - 1) / kf::gemm_mfma_tile_n();
  const int64_t T = tm_n * tn_n;
  const int64_t G = gemm_pp_workgroups(d);
  if (T <= 0 || T > (int64_t(1) << 22) || G <= 0) return -1.0;
  const double es = s.in_dtype == KF_FP8_E4M3 ? 1.0 : 2.0;
  const double a_panel = 128.0 * (double)s.K * es;
  const double b_panel = (double)kf::gemm_mfma_tile_n() * (double)s.K * es;
  double bytes = 0.0;
  std::vector<uint8_t> seen_m((size_t)tm_n * 8), seen_n((size_t)tn_n * 8);
  for (int64_t i = 0;; ++i) {
    std::fill(seen_m.begin(), seen_m.end(), 0);
    std::fill(seen_n.begin(), seen_n.end(), 0);
    bool any = false;
    for (int64_t b = 0; b < G; ++b) {
      int64_t lid;
      if ((T & 7) == 0 && (G & 7) == 0) {
        const int64_t local = i * (G >> 3) + (b >> 3);
        if (local >= (T >> 3)) continue;
        lid = (b & 7) * (T >> 3) + local;
      } else {
        lid = b + i * G;
        if (lid >= T) continue;
      }
      any = true;
      const int64_t per_group = 8 * tn_n, group = lid / per_group, first_m = group * 8;
      const int64_t gsize = std::min<int64_t>(tm_n - first_m, 8), rr = lid - group * per_group;
      const int64_t tm = first_m + rr % gsize, tn = rr / gsize, x = b & 7;
      uint8_t& fm = seen_m[(size_t)(tm * 8 + x)];
      uint8_t& fn = seen_n[(size_t)(tn * 8 + x)];
      if (!fm) bytes += a_panel;
      if (!fn) bytes += b_panel;
      fm = fn = 1;
    }
    if (!any) break;
  }
  return bytes;
}

}  // namespace

kf_status kf_autotune(kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream, int32_t reps,
                      kf_tune_result* result) {
  if (!d || !inputs || !outputs || !result) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  if (reps < 1 || reps > 1000) return fail(KF_ERR_INVALID_ARG, "reps must be in [1, 1000]");
  std::vector<kf_tuning> cand;
  const kf_tuning cur = d->tuning;
  if (d->variant == kVarGemmBf16 || d->variant == kVarGemmFp8) {
    // both store paths of the 256x256 kernel over every tile order
    for (int v : {0, 2})
      for (int remap = 1; remap >= 0; --remap)
        for (int g : {1, 2, 4, 8, 16, 32, 64}) cand.push_back(kf_tuning{g, remap, cur.wg_per_cu, v});
    // the second tile shape (its tile order is fixed: raster and XCD fields unused)
    if (d->spec.b_layout == KF_LAYOUT_KN) cand.push_back(kf_tuning{cur.raster_group, cur.xcd_remap, cur.wg_per_cu, 1});
  } else if (d->variant == kVarConv3d) {
    for (int remap = 1; remap >= 0; --remap)
      for (int wg : {2, 1}) cand.push_back(kf_tuning{cur.raster_group, remap, wg, 0});
  } else if (d->variant == kVarConvBf16 && d->conv_special) {
    for (int v : {0, 1}) cand.push_back(kf_tuning{cur.raster_group, cur.xcd_remap, cur.wg_per_cu, v});
  } else {
    cand.push_back(cur);
  }
  memset(result, 0, sizeof(*result));
  const int n = (int)std::min<size_t>(cand.size(), KF_MAX_TUNE_CANDIDATES);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    (void)hipGetLastError();
    if (e0) (void)hipEventDestroy(e0);
    return fail(KF_ERR_HIP, "hipEventCreate failed");
  }
  // The GPU's clock drifts under power management over a few milliseconds,
  // so the candidates are timed in kRounds interleaved rounds and each is
  // ranked by its median round: no candidate is favoured by when it ran.
  constexpr int kRounds = 3;
  std::vector<double> t((size_t)n * kRounds, 0.0);
  kf_status st = KF_OK;
  for (int round = 0; round < kRounds && st == KF_OK; ++round) {
    for (int c = 0; c < n && st == KF_OK; ++c) {
      d->tuning = cand[c];
      st = kf_fused_op(d, inputs, outputs, stream);  // warm-up (also validates the tensors)
      if (st != KF_OK) break;
      if (hipEventRecord(e0, hs) != hipSuccess) st = fail(KF_ERR_HIP, "hipEventRecord failed");
      for (int r = 0; r < reps && st == KF_OK; ++r) st = kf_fused_op(d, inputs, outputs, stream);
      if (st != KF_OK) break;
      float ms = 0.0f;
      if (hipEventRecord(e1, hs) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
          hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
        st = fail(KF_ERR_HIP, "timing a candidate failed: %s", hipGetErrorString(hipGetLastError()));
        break;
      }
      t[(size_t)c * kRounds + round] = (double)ms * 1e-3 / reps;
    }
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (st != KF_OK || n == 0) {
    d->tuning = cur;
    return st != KF_OK ? st : fail(KF_ERR_INVALID_ARG, "no candidate configuration");
  }
  const bool gemm = d->variant == kVarGemmBf16 || d->variant == kVarGemmFp8;
  int best = 0;
  for (int c = 0; c < n; ++c) {
    double* r = &t[(size_t)c * kRounds];
    std::sort(r, r + kRounds);
    result->config[c] = cand[c];
    result->seconds[c] = r[kRounds / 2];
    result->panel_bytes[c] = gemm ? gemm_panel_bytes(d, cand[c]) : -1.0;
    if (result->seconds[c] < result->seconds[best]) best = c;
  }
  // within 2% of the fastest time, the fewest fetched operand panels
  const double fastest = result->seconds[best];
  for (int c = 0; c < n && gemm; ++c)
    if (result->seconds[c] <= fastest * 1.02 && result->panel_bytes[c] >= 0.0 &&
        result->panel_bytes[c] < result->panel_bytes[best])
      best = c;
  result->n = n;
  result->best = best;
  d->tuning = result->config[best];
  return ok();
}

const char* kf_status_string(kf_status st) {
  switch (st) {
    case KF_OK: return "KF_OK";
    case KF_ERR_INVALID_ARG: return "KF_ERR_INVALID_ARG: invalid argument";
    case KF_ERR_SHAPE: return "KF_ERR_SHAPE: tensor shape, dtype or stride does not match the op";
    case KF_ERR_UNSUPPORTED: return "KF_ERR_UNSUPPORTED: not supported by this library";
    case KF_ERR_NO_DEVICE: return "KF_ERR_NO_DEVICE: no gfx950 device available";
    case KF_ERR_OOM: return "KF_ERR_OOM: device workspace allocation failed";
    case KF_ERR_HIP: return "KF_ERR_HIP: HIP runtime error";
    default: return "unknown kf_status";
  }
}

const char* kf_last_error(void) { return g_last_error; }

kf_status kf_create(const kf_op_spec* spec, kf_desc** out) {
  if (!out) return fail(KF_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  kf_desc* d = new (std::nothrow) kf_desc();
  if (!d) return fail(KF_ERR_OOM, "host allocation failed");
  init_desc(d);
  kf_status st = validate_and_plan(spec, d);
  if (st != KF_OK) {
    delete d;
    return st;
  }
  d->spec = *spec;
  d->chain = match_chain(spec);

  int dev = 0, cus = 0;
  st = current_device(&dev, &cus);
  if (st != KF_OK) {
    delete d;
    return st;
  }
  d->device = dev;
  d->num_cu = cus;

  d->workspace_bytes = plan_workspace_bytes(d);
  if (d->workspace_bytes && hipMalloc(&d->workspace, d->workspace_bytes) != hipSuccess) {
    (void)hipGetLastError();
    delete d;
    return fail(KF_ERR_OOM, "workspace of %zu bytes could not be allocated", d->workspace_bytes);
  }
  *out = d;
  return ok();
}

void kf_destroy(kf_desc* d) {
  if (!d) return;
  if (d->workspace) (void)hipFree(d->workspace);
  for (void* b : d->ubuf)
    if (b) (void)hipFree(b);
  delete d;
}

int32_t kf_num_inputs(const kf_desc* d) { return d ? (int32_t)d->inputs.size() : -1; }

kf_status kf_input_info(const kf_desc* d, int32_t slot, int32_t* dtype, int32_t* ndim, int64_t shape[KF_MAX_DIMS]) {
  if (!d || !dtype || !ndim || !shape) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  if (slot < 0 || slot >= (int32_t)d->inputs.size()) return fail(KF_ERR_INVALID_ARG, "slot %d out of range", slot);
  const Slot& s = d->inputs[slot];
  *dtype = s.dtype;
  *ndim = s.ndim;
  for (int i = 0; i < KF_MAX_DIMS; ++i) shape[i] = s.shape[i];
  return ok();
}

kf_status kf_output_info(const kf_desc* d, int32_t* dtype, int32_t* ndim, int64_t shape[KF_MAX_DIMS]) {
  if (!d || !dtype || !ndim || !shape) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  *dtype = d->output.dtype;
  *ndim = d->output.ndim;
  for (int i = 0; i < KF_MAX_DIMS; ++i) shape[i] = d->output.shape[i];
  return ok();
}

size_t kf_workspace_bytes(const kf_desc* d) { return d ? d->workspace_bytes : 0; }

const char* kf_kernel_name(const kf_desc* d) {
  if (!d) return "";
  if ((d->variant == kVarGemmBf16 || d->variant == kVarGemmFp8) && d->tuning.variant == 1)
    return "kf_gemm_mfma_pp128x256";
  if (d->variant == kVarConvBf16)  // the launch variant picks the kernel
    return d->tuning.variant == 2 ? "kf_conv3x3_bf16_gen"
           : d->tuning.variant == 1 ? "kf_conv3x3_bf16_w8"
                                    : "kf_conv3x3_bf16_256x128";
  return d->kernel_name;
}

kf_status kf_fused_op(const kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream) {
  return kf_fused_op_timed(d, inputs, outputs, stream, nullptr, nullptr);
}

kf_status kf_fused_op_timed(const kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream,
                            void* ev_before, void* ev_after) {
  if (!d || !inputs || !outputs) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  return run_fused(d, d->workspace, true, inputs, outputs, stream, ev_before, ev_after);
}

void kf_weights_changed(kf_desc* d) {
  if (d) d->packed_from = nullptr;
}

int64_t kf_wall_clock_hz(void) {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) {
    (void)hipGetLastError();
    return -1;
  }
  return (int64_t)khz * 1000;
}

kf_status kf_set_clock_stamps(kf_desc* d, void* stamps, int64_t workgroups) {
  if (!d) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  if (d->variant != kVarGemmBf16 && d->variant != kVarGemmFp8)
    return fail(KF_ERR_UNSUPPORTED, "clock stamps are recorded by the bf16 / fp8 GEMM kernel only");
  if (stamps != nullptr && workgroups < 1) return fail(KF_ERR_INVALID_ARG, "workgroups must be >= 1");
  if (reinterpret_cast<uintptr_t>(stamps) % 8) return fail(KF_ERR_INVALID_ARG, "stamps must be 8-byte aligned");
  d->stamps = static_cast<long long*>(stamps);
  d->stamp_cap = stamps ? workgroups : 0;
  return ok();
}

kf_status kf_fused_op_noalloc(const kf_op_spec* spec, const kf_tensor* inputs, kf_tensor* outputs, void* stream) {
  if (!spec || !inputs || !outputs) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  kf_desc d;  // the plan lives on the stack: it holds no heap memory
  init_desc(&d);
  kf_status st = validate_and_plan(spec, &d);
  if (st != KF_OK) return st;
  d.spec = *spec;
  d.chain = match_chain(spec);
  const size_t need = plan_workspace_bytes(&d);
  if (need > kf::scratch_bytes())
    return fail(KF_ERR_UNSUPPORTED,
                "this op needs %zu bytes of device scratch; kf_fused_op_noalloc's static scratch holds %zu "
                "(use kf_create / kf_fused_op)",
                need, kf::scratch_bytes());
  int dev = 0, cus = 0;
  st = current_device(&dev, &cus);
  if (st != KF_OK) return st;
  d.device = dev;
  d.num_cu = cus;
  void* ws = nullptr;
  if (need) {
    const hipError_t e = kf::scratch_address(dev, &ws);
    if (e != hipSuccess) return fail(KF_ERR_HIP, "static scratch lookup failed: %s", hipGetErrorString(e));
  }
  return run_fused(&d, ws, false, inputs, outputs, stream, nullptr, nullptr);
}

}  // extern "C"

namespace {

kf_status run_fused(const kf_desc* d, void* ws, bool ws_keeps_weights, const kf_tensor* inputs, kf_tensor* outputs,
                    void* stream, void* ev_before, void* ev_after) {
  for (size_t i = 0; i < d->inputs.size(); ++i) {
    kf_status st = check_tensor(&inputs[i], d->inputs[i], false, d->variant != kVarGemmF32);
    if (st != KF_OK) return st;
  }
  kf_status st = check_tensor(&outputs[0], d->output, true, d->variant != kVarGemmF32);
  if (st != KF_OK) return st;

  const kf_op_spec& s = d->spec;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  if (s.contraction == KF_CONV3D_3X3X3) {
    const bool tiled = conv3d_uses_tiled(d, inputs);
    if (!tiled && d->conv3d_split < s.n_ops) {
      // the general kernel with the leading ops fused, then one kernel per
      // remaining op through the descriptor's intermediate buffers
      if (!ws_keeps_weights)
        return fail(KF_ERR_UNSUPPORTED,
                    "this Conv3d chain takes intermediate buffers outside the tiled kernel's family "
                    "(use kf_create / kf_fused_op)");
      return run_chain_split(d, inputs, outputs, stream, d->conv3d_split, ev_before, ev_after);
    }
    const kf::Conv3dArgs a = conv3d_args(d, inputs, outputs[0].data, conv3d_pool_count(s));
    if (tiled ? a.tiles == 0 : kf::conv3d_gen_tiles(s.batch, s.depth, s.height, s.width, s.cout) == 0) return ok();
    hipError_t e = conv3d_pack(d, ws, ws_keeps_weights, tiled, inputs[1].data, hs);
    if (e == hipSuccess && ev_before) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_before), hs);
    if (e == hipSuccess)
      e = tiled ? kf::launch_conv3d_bf16(a, ws, d->chain, hs)
                : kf::launch_conv3d_gen(conv3d_gen_args(d, inputs, outputs[0].data, d->prog), ws, hs);
    if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
    if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return ok();
  }
  if (s.contraction == KF_ROWWISE) {
    if (s.M == 0) return ok();
    kf::RowArgs r;
    memset(&r, 0, sizeof(r));
    r.a = inputs[0].data;
    r.M = s.M;
    r.N = s.N;
    r.lda = inputs[0].stride[0];
    r.in_bf16 = s.in_dtype == KF_BF16;
    r.prog = d->prog;
    r.gn_group = d->gn_group;
    size_t slot = 1;
    for (int i = 0; i < s.n_ops; ++i) {
      const int k = s.ops[i].kind;
      if (k == KF_OP_BIAS) r.bias = static_cast<const float*>(inputs[slot++].data);
      if (k == KF_OP_GROUPNORM) {
        r.gamma = static_cast<const float*>(inputs[slot++].data);
        r.beta = static_cast<const float*>(inputs[slot++].data);
      }
      if (k == KF_OP_RESIDUAL_ADD) {
        r.residual = inputs[slot].data;
        r.ldr = inputs[slot].stride[0];
        r.residual_bf16 = inputs[slot].dtype == KF_BF16;
        ++slot;
      }
      if (k == KF_OP_ROW_CROSS_ENTROPY) r.targets = static_cast<const int32_t*>(inputs[slot++].data);
    }
    r.out = outputs[0].data;
    r.ldo = outputs[0].ndim == 2 ? outputs[0].stride[0] : 1;
    r.out_bf16 = outputs[0].dtype == KF_BF16;
    hipError_t e = hipSuccess;
    if (ev_before) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_before), hs);
    if (e == hipSuccess) e = kf::launch_rowwise(r, d->chain, hs);
    if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
    if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return ok();
  }
  if (s.contraction == KF_GEMM) {
    if (s.M == 0) return ok();
    kf::GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.a = inputs[0].data;
    a.b = inputs[1].data;
    a.M = s.M;
    a.N = s.N;
    a.K = s.K;
    a.lda = s.K ? inputs[0].stride[0] : 8;
    a.ldb = s.K ? inputs[1].stride[0] : 8;
    a.prog = d->prog;
    a.scale = 1.0f;
    a.gn_group = d->gn_group;
    a.red_index = d->red_index;
    size_t slot = 2;
    for (int i = 0; i < s.n_ops; ++i) {
      const int k = s.ops[i].kind;
      if (k == KF_OP_BIAS) a.bias = static_cast<const float*>(inputs[slot++].data);
      if (k == KF_OP_GROUPNORM) {
        a.gamma = static_cast<const float*>(inputs[slot++].data);
        a.beta = static_cast<const float*>(inputs[slot++].data);
      }
      if (k == KF_OP_RESIDUAL_ADD) {
        a.residual = inputs[slot].data;
        a.ldr = inputs[slot].stride[0];
        a.residual_bf16 = inputs[slot].dtype == KF_BF16;
        ++slot;
      }
      if (k == KF_OP_ROW_CROSS_ENTROPY) a.targets = static_cast<const int32_t*>(inputs[slot++].data);
    }
    a.out = outputs[0].data;
    a.ldo = outputs[0].ndim == 2 ? outputs[0].stride[0] : 1;
    a.out_bf16 = outputs[0].dtype == KF_BF16;
    a.partials = ws;
    if (a.targets)  // the target logits follow the (max, sum) partials
      a.tlogit = reinterpret_cast<float*>(static_cast<unsigned char*>(ws) + (size_t)std::max<int64_t>(s.M, 1) * d->tiles_n * 8);
    a.raster_group = d->tuning.raster_group;
    a.xcd_remap = d->tuning.xcd_remap;
    a.stage_out = d->tuning.variant == 2;
    a.stamps = d->stamps;
    a.stamp_cap = d->stamp_cap;
    const bool nk = s.b_layout == KF_LAYOUT_NK;
    hipError_t e = hipSuccess;
    if (ev_before) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_before), hs);
    if (e != hipSuccess) return fail(KF_ERR_HIP, "hipEventRecord failed: %s", hipGetErrorString(e));
    if (d->variant == kVarGemmF32) {
      e = kf::launch_gemm_f32(a, nk, hs);
      if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
    } else {
      const int64_t es = elem_size(s.in_dtype);
      // the K loop addresses up to four K-steps (at most 256 k) past K, all out of range
      if (!fits_31(256 * a.lda * es) || !fits_31((nk ? 256 * a.ldb : (s.K + 256) * a.ldb) * es) ||
          !fits_31(256 * a.ldo * 4) || (a.residual && !fits_31(256 * a.ldr * 4)))
        return fail(KF_ERR_UNSUPPORTED, "operand extent too large for 32-bit buffer offsets");
      if (d->variant == kVarGemmFp8) a.scale = s.scale_a * s.scale_b;  // fl(s_a * s_b), applied to the fp32 accumulator
      e = kf::launch_gemm_mfma(a, d->variant == kVarGemmFp8, d->epi_shape, d->chain, hs, nk, gemm_pp_workgroups(d));
      if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
      if (e == hipSuccess && d->row_kind)
        e = kf::launch_row_finish(d->row_kind == KF_OP_ROW_SOFTMAX, ws, d->tiles_n, s.M, s.N, a.out,
                                  a.ldo, a.out_bf16 != 0, hs, a.targets, a.tlogit);
    }
    if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return ok();
  }
  // CONV2D_3X3
  if (s.batch == 0) return ok();
  kf::ConvArgs c;
  memset(&c, 0, sizeof(c));
  c.x = inputs[0].data;
  c.w = inputs[1].data;
  c.batch = s.batch;
  c.cin = s.cin;
  c.H = s.height;
  c.W = s.width;
  c.cout = s.cout;
  c.tiles = (int32_t)(s.batch * (s.height / 2));
  c.grid = d->num_cu;
  c.variant = d->tuning.variant;
  c.prog = d->prog;
  for (int i = 0; i < s.n_ops; ++i) {
    if (s.ops[i].kind == KF_OP_BIAS) c.bias = static_cast<const float*>(inputs[2].data);
    if (s.ops[i].kind == KF_OP_MAXPOOL2X2) {
      c.pool = 1;
      c.pool_index = i;
    }
  }
  c.out = outputs[0].data;
  c.out_bf16 = 1;
  hipError_t e = hipSuccess;
  if (!ws_keeps_weights || d->packed_from != inputs[1].data) {
    d->packed_from = nullptr;
    e = kf::launch_conv_pack(c, ws, hs);
    if (e == hipSuccess && ws_keeps_weights) d->packed_from = inputs[1].data;
  }
  if (e == hipSuccess && ev_before) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_before), hs);
  if (e == hipSuccess) e = kf::launch_conv_bf16(c, ws, d->chain, hs);
  if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
  if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

namespace {

// Run plan d as its contraction with ops [0, prefix) fused (prefix > 0 only
// for the general conv3d kernel: BIAS and element-wise ops), then one kernel
// per remaining op, every intermediate stored in bf16 (fp32 for an fp32
// chain) in the descriptor's two buffers, allocated on first use.  prefix 0
// is the unfused comparator.  ev_before / ev_after bracket the contraction.
kf_status run_chain_split(const kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream, int prefix,
                          void* ev_before, void* ev_after) {
  const kf_op_spec& s = d->spec;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const bool gemm = s.contraction == KF_GEMM;
  const bool rowwise = s.contraction == KF_ROWWISE;
  const bool conv3d = s.contraction == KF_CONV3D_3X3X3;
  const bool rows = gemm || rowwise;  // an [M, N] intermediate
  if ((rows && s.M == 0) || (!rows && s.batch == 0)) return ok();
  const int n_rest = s.n_ops - prefix;

  // intermediates: bf16 (fp32 for an fp32 chain), full contraction size
  const bool ibf16 = rowwise ? s.in_dtype == KF_BF16 : d->variant != kVarGemmF32;
  const int64_t n_full = rows     ? s.M * s.N
                         : conv3d ? s.batch * s.cout * (s.depth - 2) * (s.height - 2) * (s.width - 2)
                                  : s.batch * s.cout * s.height * s.width;
  const size_t need = (size_t)n_full * (ibf16 ? 2 : 4);
  if (n_rest > 0 && d->ubuf_bytes < need) {
    for (void*& b : d->ubuf) {
      if (b) (void)hipFree(b);
      b = nullptr;
      if (hipMalloc(&b, need) != hipSuccess) {
        (void)hipGetLastError();
        d->ubuf_bytes = 0;
        return fail(KF_ERR_OOM, "unfused intermediates of %zu bytes could not be allocated", need);
      }
    }
    d->ubuf_bytes = need;
  }

  // 1. the contraction alone (empty op list), into the first buffer -- or
  //    straight into the output when there are no ops
  void* out = outputs[0].data;
  const bool out_bf16 = outputs[0].dtype == KF_BF16;
  void* cur = n_rest ? d->ubuf[0] : out;
  bool cur_bf16 = n_rest ? ibf16 : out_bf16;
  hipError_t e = hipSuccess;
  size_t slot = 2;
  for (int i = 0; i < prefix; ++i) slot += s.ops[i].kind == KF_OP_BIAS;  // tensors the fused prefix takes
  if (ev_before) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_before), hs);
  if (rowwise) {
    // no contraction: the first op reads A itself (an empty list copies it)
    slot = 1;
    cur = inputs[0].data;
    cur_bf16 = s.in_dtype == KF_BF16;
    if (!s.n_ops) e = kf::launch_unfused_elementwise(cur, cur_bf16, out, out_bf16, n_full, 0, 0.f, 0.f, nullptr, 1, 1, hs);
  } else if (gemm) {
    kf::GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.a = inputs[0].data;
    a.b = inputs[1].data;
    a.M = s.M;
    a.N = s.N;
    a.K = s.K;
    a.lda = s.K ? inputs[0].stride[0] : 8;
    a.ldb = s.K ? inputs[1].stride[0] : 8;
    a.scale = d->variant == kVarGemmFp8 ? s.scale_a * s.scale_b : 1.0f;
    a.out = cur;
    a.ldo = s.n_ops ? s.N : (outputs[0].ndim == 2 ? outputs[0].stride[0] : 1);
    a.out_bf16 = cur_bf16;
    a.red_index = 0;
    a.raster_group = d->tuning.raster_group;
    a.xcd_remap = d->tuning.xcd_remap;
    const bool nk = s.b_layout == KF_LAYOUT_NK;
    if (d->variant != kVarGemmF32) {
      const int64_t es = elem_size(s.in_dtype);
      // as in the fused path: 32-bit buffer offsets over up to 256 rows / k past the tile
      if (!fits_31(256 * a.lda * es) || !fits_31((nk ? 256 * a.ldb : (s.K + 256) * a.ldb) * es) ||
          !fits_31(256 * a.ldo * 4))
        return fail(KF_ERR_UNSUPPORTED, "operand extent too large for 32-bit buffer offsets");
    }
    e = d->variant == kVarGemmF32 ? kf::launch_gemm_f32(a, nk, hs)
                                  : kf::launch_gemm_mfma(a, d->variant == kVarGemmFp8, kf::kEpiPlain, 1, hs, nk,
                                                         gemm_pp_workgroups(d));
  } else if (conv3d) {
    // the convolution (with the fused prefix): every conv output position, NCDHW
    const bool tiled = prefix == 0 && conv3d_uses_tiled(d, inputs);
    const kf::Conv3dArgs a = conv3d_args(d, inputs, cur, 0);
    if (e == hipSuccess) e = conv3d_pack(d, d->workspace, true, tiled, inputs[1].data, hs);
    if (e == hipSuccess && tiled && a.tiles) e = kf::launch_conv3d_bf16(a, d->workspace, 1, hs);
    if (e == hipSuccess && !tiled) {
      kf::EpiProgram pre;
      memset(&pre, 0, sizeof(pre));
      pre.n = prefix;
      for (int i = 0; i < prefix; ++i) pre.op[i] = d->prog.op[i];
      e = kf::launch_conv3d_gen(conv3d_gen_args(d, inputs, cur, pre), d->workspace, hs);
    }
  } else {
    kf::ConvArgs c;
    memset(&c, 0, sizeof(c));
    c.x = inputs[0].data;
    c.w = inputs[1].data;
    c.batch = s.batch;
    c.cin = s.cin;
    c.H = s.height;
    c.W = s.width;
    c.cout = s.cout;
    c.tiles = (int32_t)(s.batch * (s.height / 2));
    c.grid = d->num_cu;
    c.variant = d->tuning.variant;
    c.out = cur;
    c.out_bf16 = 1;
    if (d->packed_from != inputs[1].data) {
      d->packed_from = nullptr;
      e = kf::launch_conv_pack(c, d->workspace, hs);
      if (e == hipSuccess) d->packed_from = inputs[1].data;
    }
    if (e == hipSuccess) e = kf::launch_conv_bf16(c, d->workspace, 0, hs);
  }
  if (e == hipSuccess && ev_after) e = hipEventRecord(reinterpret_cast<hipEvent_t>(ev_after), hs);
  if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));

  // 2. one kernel per op, ping-ponging between the buffers; the last op
  //    writes the output
  int64_t n = n_full;
  int64_t dd = conv3d ? s.depth - 2 : 1, hh = conv3d ? s.height - 2 : s.height, ww = conv3d ? s.width - 2 : s.width;
  int which = 0;
  for (int i = prefix; i < s.n_ops && e == hipSuccess; ++i) {
    const kf_op& op = s.ops[i];
    const bool last = i == s.n_ops - 1;
    void* dst = last ? out : d->ubuf[which ^ 1];
    const bool dst_bf16 = last ? out_bf16 : ibf16;
    switch (op.kind) {
      case KF_OP_BIAS: {
        const float* bias = static_cast<const float*>(inputs[slot++].data);
        const int64_t fdiv = rows ? 1 : dd * hh * ww, fmod = rows ? s.N : s.cout;
        e = kf::launch_unfused_elementwise(cur, cur_bf16, dst, dst_bf16, n, op.kind, 0.f, 0.f, bias, fdiv, fmod, hs);
        break;
      }
      case KF_OP_RESIDUAL_ADD: {
        const kf_tensor& r = inputs[slot++];
        e = kf::launch_unfused_residual(cur, cur_bf16, r.data, r.dtype == KF_BF16, dst, dst_bf16, n, hs);
        break;
      }
      case KF_OP_GROUPNORM: {
        const float* gamma = static_cast<const float*>(inputs[slot++].data);
        const float* beta = static_cast<const float*>(inputs[slot++].data);
        e = kf::launch_unfused_groupnorm(cur, cur_bf16, dst, dst_bf16, s.M, s.N, op.groups, op.p0, gamma, beta, hs);
        break;
      }
      case KF_OP_ROW_SOFTMAX:
      case KF_OP_ROW_LOGSUMEXP:
        e = kf::launch_unfused_rowop(cur, cur_bf16, dst, dst_bf16, s.M, s.N, op.kind, nullptr, hs);
        break;
      case KF_OP_ROW_CROSS_ENTROPY:
        e = kf::launch_unfused_rowop(cur, cur_bf16, dst, dst_bf16, s.M, s.N, op.kind,
                                     static_cast<const int32_t*>(inputs[slot++].data), hs);
        break;
      case KF_OP_CHANNEL_SOFTMAX:
        e = kf::launch_unfused_channel_softmax(cur, cur_bf16, dst, dst_bf16, s.batch, (int)s.cout, dd * hh * ww, hs);
        break;
      case KF_OP_MAXPOOL3D_2:
        e = kf::launch_unfused_maxpool3d(cur, cur_bf16, dst, dst_bf16, s.batch * s.cout, (int)dd, (int)hh, (int)ww, hs);
        dd /= 2;
        hh /= 2;
        ww /= 2;
        n = s.batch * s.cout * dd * hh * ww;
        break;
      case KF_OP_MAXPOOL2X2:
        e = kf::launch_unfused_maxpool(cur, cur_bf16, dst, dst_bf16, s.batch * s.cout, (int)hh, (int)ww, hs);
        hh /= 2;
        ww /= 2;
        n = s.batch * s.cout * hh * ww;
        break;
      default:
        e = kf::launch_unfused_elementwise(cur, cur_bf16, dst, dst_bf16, n, op.kind, op.p0, op.p1, nullptr, 1, 1, hs);
        break;
    }
    cur = dst;
    cur_bf16 = dst_bf16;
    which ^= 1;
  }
  if (e != hipSuccess) return fail(KF_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

kf_status kf_unfused_op(const kf_desc* d, const kf_tensor* inputs, kf_tensor* outputs, void* stream) {
  if (!d || !inputs || !outputs) return fail(KF_ERR_INVALID_ARG, "NULL argument");
  const bool vec16 = d->variant != kVarGemmF32;
  for (size_t i = 0; i < d->inputs.size(); ++i) {
    kf_status st = check_tensor(&inputs[i], d->inputs[i], false, vec16);
    if (st != KF_OK) return st;
  }
  kf_status st = check_tensor(&outputs[0], d->output, true, vec16);
  if (st != KF_OK) return st;
  const kf_op_spec& s = d->spec;
  const bool rowwise = s.contraction == KF_ROWWISE;
  const bool rows = s.contraction == KF_GEMM || rowwise;  // an [M, N] intermediate
  if ((rows && s.M == 0) || (!rows && s.batch == 0)) return ok();
  // the per-op kernels index [M, N] tensors as contiguous rows
  if (rowwise && inputs[0].stride[0] != s.N)
    return fail(KF_ERR_UNSUPPORTED, "the unfused ROWWISE chain needs A with row stride N");
  if (rows && s.n_ops) {
    for (int i = 0; i < s.n_ops; ++i)
      if (s.ops[i].kind == KF_OP_GROUPNORM && s.M * s.ops[i].groups >= kMaxRowLaunch)
        return fail(KF_ERR_UNSUPPORTED, "the unfused GroupNorm supports M * groups < %lld", (long long)kMaxRowLaunch);
    for (size_t i = 0; i < d->inputs.size(); ++i)
      if (strcmp(d->inputs[i].name, "residual") == 0 && inputs[i].stride[0] != s.N)
        return fail(KF_ERR_UNSUPPORTED, "the unfused chain needs a residual with row stride N");
    if (outputs[0].ndim == 2 && outputs[0].stride[0] != s.N)
      return fail(KF_ERR_UNSUPPORTED, "the unfused chain needs an output with row stride N");
  }

  return run_chain_split(d, inputs, outputs, stream, 0, nullptr, nullptr);
}

}  // extern "C"
