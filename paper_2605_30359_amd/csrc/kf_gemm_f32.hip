// fp32 GEMM + element-wise epilogue (true fp32 products, fp32 accumulation).
//
// The small Linear + bias + activation operator (the paper's "matmul + relu"
// fusion example, Appendix A) is latency bound: at [32,256] x [256,512] it is
// 8.4 MFLOP, 64 multiply-adds per lane if spread over the whole chip.  So the
// kernel spreads it that way: an 8 x 8 output tile per 256-thread workgroup
// (256 workgroups for that shape), the tile's 8 x 256 slice of x and 256 x 8
// slice of W staged in LDS per 256-deep K chunk, each of the 4 waves summing
// a 64-deep quarter of the chunk for all 64 outputs (one per lane), then the
// four partial sums added in wave order, the op list applied and one store.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {
constexpr int TM = 8, TN = 8, KC = 256, NT = 256;
constexpr int XP = KC + 4;  // x row pitch in floats: 16-byte aligned rows, 8 rows on distinct banks
}  // namespace

__global__ __launch_bounds__(NT) void kf_gemm_f32_8x8(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) float xs[TM * XP];
  __shared__ float ws[KC * TN];
  __shared__ float part[4 * 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t m0 = (int64_t)blockIdx.y * TM;
  const int64_t n0 = (int64_t)blockIdx.x * TN;
  const float* A = reinterpret_cast<const float*>(p.a);
  const float* B = reinterpret_cast<const float*>(p.b);
  const bool b_nk = p.ldb < 0;  // sign flags the NK layout; |ldb| is the stride
  const int64_t ldb = b_nk ? -p.ldb : p.ldb;
  const int r = lane >> 3, c = lane & 7;  // this lane's output (m0 + r, n0 + c)
  const int64_t m = m0 + r, n = n0 + c;
  const bool out_ok = m < p.M && n < p.N;
  // the epilogue's tensor operands of this lane's output, requested now so
  // that their latency overlaps the operand loads instead of following them
  float bias_v = 0.0f, res_v = 0.0f;
  if (wave == 0 && out_ok) {
    if (p.bias) bias_v = p.bias[n];
    if (p.residual)
      res_v = p.residual_bf16
                  ? __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(p.residual)[m * p.ldr + n] << 16)
                  : reinterpret_cast<const float*>(p.residual)[m * p.ldr + n];
  }

  float acc = 0.0f;
  for (int64_t k0 = 0; k0 < p.K; k0 += KC) {
    // x slice [8][256]: thread t loads column k0 + t of all 8 rows
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t gm = m0 + i, gk = k0 + tid;
      xs[i * XP + tid] = (gm < p.M && gk < p.K) ? A[gm * p.lda + gk] : 0.0f;
    }
    // W slice [256][8]: coalesced along n (KN) or along k (NK)
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      int k, n;
      if (b_nk) {
        k = tid;
        n = i;
      } else {
        k = (tid >> 3) + 32 * i;
        n = tid & 7;
      }
      const int64_t gk = k0 + k, gn = n0 + n;
      float w = 0.0f;
      if (gk < p.K && gn < p.N) w = b_nk ? B[gn * ldb + gk] : B[gk * ldb + gn];
      ws[k * TN + n] = w;
    }
    __syncthreads();
    const float* xr = xs + r * XP + wave * 64;
    const float* wc = ws + wave * 64 * TN + c;
#pragma unroll 4
    for (int kk = 0; kk < 64; kk += 4) {
      const f32x4 x4 = *reinterpret_cast<const f32x4*>(xr + kk);
      acc = fmaf(x4[0], wc[(kk + 0) * TN], acc);
      acc = fmaf(x4[1], wc[(kk + 1) * TN], acc);
      acc = fmaf(x4[2], wc[(kk + 2) * TN], acc);
      acc = fmaf(x4[3], wc[(kk + 3) * TN], acc);
    }
    __syncthreads();
  }
  part[wave * 64 + lane] = acc;
  __syncthreads();
  if (wave != 0) return;

  if (!out_ok) return;
  float x = ((part[lane] + part[64 + lane]) + part[128 + lane]) + part[192 + lane];
  x *= p.scale;
  for (int o = 0; o < p.prog.n; ++o) {
    const EpiOp op = p.prog.op[o];
    if (op.kind == KF_OP_BIAS) {
      x += bias_v;
    } else if (op.kind == KF_OP_RESIDUAL_ADD) {
      x += res_v;
    } else {
      x = apply_elementwise(op.kind, op.p0, op.p1, x);
    }
  }
  if (p.out_bf16)
    reinterpret_cast<uint16_t*>(p.out)[m * p.ldo + n] = (uint16_t)f32_to_bf16_rne(x);
  else
    reinterpret_cast<float*>(p.out)[m * p.ldo + n] = x;
}

hipError_t launch_gemm_f32(const GemmArgs& args, bool b_nk, hipStream_t stream) {
  GemmArgs p = args;
  if (b_nk) p.ldb = -p.ldb;
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  const dim3 grid((unsigned)((p.N + TN - 1) / TN), (unsigned)((p.M + TM - 1) / TM));
  hipLaunchKernelGGL(kf_gemm_f32_8x8, grid, dim3(NT), 0, stream, p);
  return hipGetLastError();
}

}  // namespace kf
