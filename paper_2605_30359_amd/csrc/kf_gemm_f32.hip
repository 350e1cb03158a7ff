// fp32 GEMM + element-wise epilogue (true fp32 products, fp32 accumulation).
//
// The small Linear + bias + activation operator (the paper's "matmul + relu"
// fusion example, Appendix A) is launch-latency bound: at [32,256] x
// [256,512] it is 8.4 MFLOP, so the kernel is a plain LDS-tiled FMA kernel
// with a 32 x 64 output tile per 256-thread workgroup (8 rows x 1 column per
// thread) and the op list applied to each output before the only store.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {
constexpr int TM = 32, TN = 64, TK = 32, NT = 256;
}

__global__ __launch_bounds__(NT) void kf_gemm_f32_32x64(GemmArgs p) {
  __shared__ float xs[TM][TK + 1];
  __shared__ float ws[TK][TN];
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.y * TM;
  const int64_t n0 = (int64_t)blockIdx.x * TN;
  const int col = tid & (TN - 1);
  const int rbase = (tid >> 6) * 8;
  const float* A = reinterpret_cast<const float*>(p.a);
  const float* B = reinterpret_cast<const float*>(p.b);
  const bool b_nk = p.ldb < 0;  // sign flags the NK layout; |ldb| is the stride
  const int64_t ldb = b_nk ? -p.ldb : p.ldb;

  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.0f;

  for (int64_t k0 = 0; k0 < p.K; k0 += TK) {
    // x tile: 32 x 32 -> 4 per thread
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = tid + NT * i;
      const int r = e / TK, k = e % TK;
      const int64_t gm = m0 + r, gk = k0 + k;
      xs[r][k] = (gm < p.M && gk < p.K) ? A[gm * p.lda + gk] : 0.0f;
    }
    // w tile: 32 x 64 -> 8 per thread
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int e = tid + NT * i;
      const int k = e / TN, n = e % TN;
      const int64_t gk = k0 + k, gn = n0 + n;
      float w = 0.0f;
      if (gk < p.K && gn < p.N) w = b_nk ? B[gn * ldb + gk] : B[gk * ldb + gn];
      ws[k][n] = w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      const float w = ws[k][col];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = fmaf(xs[rbase + i][k], w, acc[i]);
    }
    __syncthreads();
  }

  const int64_t n = n0 + col;
  if (n >= p.N) return;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t m = m0 + rbase + i;
    if (m >= p.M) continue;
    float x = acc[i] * p.scale;
    for (int o = 0; o < p.prog.n; ++o) {
      const EpiOp op = p.prog.op[o];
      if (op.kind == KF_OP_BIAS) {
        x += p.bias[n];
      } else if (op.kind == KF_OP_RESIDUAL_ADD) {
        if (p.residual_bf16)
          x += __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(p.residual)[m * p.ldr + n] << 16);
        else
          x += reinterpret_cast<const float*>(p.residual)[m * p.ldr + n];
      } else {
        x = apply_elementwise(op.kind, op.p0, op.p1, x);
      }
    }
    if (p.out_bf16)
      reinterpret_cast<uint16_t*>(p.out)[m * p.ldo + n] = (uint16_t)f32_to_bf16_rne(x);
    else
      reinterpret_cast<float*>(p.out)[m * p.ldo + n] = x;
  }
}

hipError_t launch_gemm_f32(const GemmArgs& args, bool b_nk, hipStream_t stream) {
  GemmArgs p = args;
  if (b_nk) p.ldb = -p.ldb;
  const dim3 grid((unsigned)((p.N + TN - 1) / TN), (unsigned)((p.M + TM - 1) / TM));
  hipLaunchKernelGGL(kf_gemm_f32_32x64, grid, dim3(NT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace kf
