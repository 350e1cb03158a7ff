// The unfused comparator: one kernel per op, every intermediate stored to
// device memory (bf16, or fp32 for fp32 chains) -- the one-kernel-per-operator
// form that operator fusion removes (Appendix A, "Operator Fusion"; the
// paper's speedups are measured against such eager operator chains).  The
// contraction itself reuses the fused kernels with an empty op list.
//
// All kernels here are memory-bound: 16-byte loads and stores, fp32 math.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

__device__ __forceinline__ float load_elem(const void* p, int64_t i, bool bf16) {
  return bf16 ? __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(p)[i] << 16)
              : reinterpret_cast<const float*>(p)[i];
}
__device__ __forceinline__ void store_elem(void* p, int64_t i, float v, bool bf16) {
  if (bf16)
    reinterpret_cast<uint16_t*>(p)[i] = (uint16_t)f32_to_bf16_rne(v);
  else
    reinterpret_cast<float*>(p)[i] = v;
}

// block-wide sum / max over 256 threads
template <bool IS_MAX>
__device__ __forceinline__ float block_reduce(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float y = __shfl_xor(v, o, 64);
    v = IS_MAX ? fmaxf(v, y) : v + y;
  }
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < 4; ++i) r = IS_MAX ? fmaxf(r, red[i]) : r + red[i];
  return r;
}

}  // namespace

// out[i] = op(in[i]); BIAS adds bias[(i / fdiv) % fmod] (feature index).
// 8 elements per thread when both sides are bf16 and n % 8 == 0.
__global__ __launch_bounds__(256) void kf_unfused_elementwise(const void* in, int in_bf16, void* out, int out_bf16,
                                                              int64_t n, int kind, float p0, float p1,
                                                              const float* bias, int64_t fdiv, int64_t fmod) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  if (in_bf16 && out_bf16 && (n & 7) == 0) {
    const int64_t nv = n >> 3;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < nv; v += stride) {
      u32x4 w = reinterpret_cast<const u32x4*>(in)[v];
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float a = bf16_lo(w[e]), b = bf16_hi(w[e]);
        if (kind == KF_OP_BIAS) {
          const int64_t i = v * 8 + e * 2;
          a += bias[(i / fdiv) % fmod];
          b += bias[((i + 1) / fdiv) % fmod];
        } else {
          a = apply_elementwise(kind, p0, p1, a);
          b = apply_elementwise(kind, p0, p1, b);
        }
        o[e] = pack_bf16x2(a, b);
      }
      reinterpret_cast<u32x4*>(out)[v] = o;
    }
    return;
  }
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    float a = load_elem(in, i, in_bf16);
    a = kind == KF_OP_BIAS ? a + bias[(i / fdiv) % fmod] : apply_elementwise(kind, p0, p1, a);
    store_elem(out, i, a, out_bf16);
  }
}

// out = in + residual (same shape)
__global__ __launch_bounds__(256) void kf_unfused_residual(const void* in, int in_bf16, const void* res, int res_bf16,
                                                           void* out, int out_bf16, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    store_elem(out, i, load_elem(in, i, in_bf16) + load_elem(res, i, res_bf16), out_bf16);
}

// GroupNorm over rows of N features in groups of gw: one workgroup per
// (row, group); mean, then biased variance of the deviations, then the affine.
__global__ __launch_bounds__(256) void kf_unfused_groupnorm(const void* in, int in_bf16, void* out, int out_bf16,
                                                            int64_t N, int gw, float eps, const float* gamma,
                                                            const float* beta) {
  __shared__ float red[4];
  const int groups = (int)(N / gw);
  const int64_t row = blockIdx.x / groups;
  const int g = blockIdx.x % groups;
  const int64_t base = row * N + (int64_t)g * gw;
  float s = 0.0f;
  for (int j = threadIdx.x; j < gw; j += 256) s += load_elem(in, base + j, in_bf16);
  const float mean = block_reduce<false>(s, red) / (float)gw;
  float q = 0.0f;
  for (int j = threadIdx.x; j < gw; j += 256) {
    const float d = load_elem(in, base + j, in_bf16) - mean;
    q += d * d;
  }
  const float rs = rsqrtf(block_reduce<false>(q, red) / (float)gw + eps);
  for (int j = threadIdx.x; j < gw; j += 256) {
    const int64_t c = (int64_t)g * gw + j;
    store_elem(out, base + j, (load_elem(in, base + j, in_bf16) - mean) * rs * gamma[c] + beta[c], out_bf16);
  }
}

// Row softmax / logsumexp over N columns: one workgroup per row.
__global__ __launch_bounds__(256) void kf_unfused_rowop(const void* in, int in_bf16, void* out, int out_bf16,
                                                        int64_t N, int softmax) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const int64_t base = row * N;
  float m = -INFINITY;
  for (int64_t j = threadIdx.x; j < N; j += 256) m = fmaxf(m, load_elem(in, base + j, in_bf16));
  m = block_reduce<true>(m, red);
  float s = 0.0f;
  for (int64_t j = threadIdx.x; j < N; j += 256) s += fexp(load_elem(in, base + j, in_bf16) - m);
  s = block_reduce<false>(s, red);
  if (!softmax) {
    if (threadIdx.x == 0) reinterpret_cast<float*>(out)[row] = m + logf(s);
    return;
  }
  const float inv = 1.0f / s;
  for (int64_t j = threadIdx.x; j < N; j += 256)
    store_elem(out, base + j, fexp(load_elem(in, base + j, in_bf16) - m) * inv, out_bf16);
}

// MaxPool2d(2, 2) on [planes][H][W] -> [planes][H/2][W/2]
__global__ __launch_bounds__(256) void kf_unfused_maxpool(const void* in, int in_bf16, void* out, int out_bf16,
                                                          int64_t planes, int H, int W) {
  const int Ho = H / 2, Wo = W / 2;
  const int64_t n = planes * Ho * Wo;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t pl = i / ((int64_t)Ho * Wo);
    const int r = (int)(i % ((int64_t)Ho * Wo));
    const int ph = r / Wo, pw = r % Wo;
    const int64_t b = (pl * H + 2 * ph) * W + 2 * pw;
    const float v = fmaxf(fmaxf(load_elem(in, b, in_bf16), load_elem(in, b + 1, in_bf16)),
                          fmaxf(load_elem(in, b + W, in_bf16), load_elem(in, b + W + 1, in_bf16)));
    store_elem(out, i, v, out_bf16);
  }
}

// Softmax over the channel axis of an NCDHW tensor, one thread per (image,
// position): consecutive threads take consecutive positions, so every read
// of one channel plane is coalesced.  Three passes over the channels (max,
// sum of exponentials, normalised store), as torch.softmax(h, dim=1) does.
__global__ __launch_bounds__(256) void kf_unfused_channel_softmax(const void* in, int in_bf16, void* out,
                                                                  int out_bf16, int64_t batch, int C,
                                                                  int64_t S) {
  const int64_t n = batch * S;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t b = (i / S) * C * S + i % S;
    float m = -INFINITY;
    for (int c = 0; c < C; ++c) m = fmaxf(m, load_elem(in, b + c * S, in_bf16));
    float sum = 0.0f;
    for (int c = 0; c < C; ++c) sum += fexp(load_elem(in, b + c * S, in_bf16) - m);
    const float inv = 1.0f / sum;
    for (int c = 0; c < C; ++c) store_elem(out, b + c * S, fexp(load_elem(in, b + c * S, in_bf16) - m) * inv, out_bf16);
  }
}

// MaxPool3d(2), stride 2, floor mode, over [planes][D][H][W].
__global__ __launch_bounds__(256) void kf_unfused_maxpool3d(const void* in, int in_bf16, void* out, int out_bf16,
                                                            int64_t planes, int D, int H, int W) {
  const int Do = D / 2, Ho = H / 2, Wo = W / 2;
  const int64_t per = (int64_t)Do * Ho * Wo;
  const int64_t n = planes * per;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t pl = i / per;
    const int r = (int)(i % per);
    const int pd = r / (Ho * Wo), ph = (r / Wo) % Ho, pw = r % Wo;
    float v = -INFINITY;
#pragma unroll
    for (int dd = 0; dd < 2; ++dd)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int64_t b = ((pl * D + 2 * pd + dd) * H + 2 * ph + hh) * W + 2 * pw;
        v = fmaxf(v, fmaxf(load_elem(in, b, in_bf16), load_elem(in, b + 1, in_bf16)));
      }
    store_elem(out, i, v, out_bf16);
  }
}

static unsigned grid_for(int64_t n) {
  const int64_t g = (n + 255) / 256;
  return (unsigned)(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

hipError_t launch_unfused_elementwise(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t n, int kind,
                                      float p0, float p1, const float* bias, int64_t fdiv, int64_t fmod,
                                      hipStream_t stream) {
  const int64_t work = (in_bf16 && out_bf16 && (n & 7) == 0) ? n / 8 : n;
  hipLaunchKernelGGL(kf_unfused_elementwise, dim3(grid_for(work)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, n, kind, p0, p1, bias, fdiv, fmod);
  return hipGetLastError();
}

hipError_t launch_unfused_residual(const void* in, bool in_bf16, const void* res, bool res_bf16, void* out,
                                   bool out_bf16, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(kf_unfused_residual, dim3(grid_for(n)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, res,
                     res_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, n);
  return hipGetLastError();
}

hipError_t launch_unfused_groupnorm(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                    int groups, float eps, const float* gamma, const float* beta,
                                    hipStream_t stream) {
  hipLaunchKernelGGL(kf_unfused_groupnorm, dim3((unsigned)(rows * groups)), dim3(256), 0, stream, in,
                     in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, N, (int)(N / groups), eps, gamma, beta);
  return hipGetLastError();
}

hipError_t launch_unfused_rowop(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                bool softmax, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(kf_unfused_rowop, dim3((unsigned)rows), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, N, softmax ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_unfused_maxpool(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int H,
                                  int W, hipStream_t stream) {
  hipLaunchKernelGGL(kf_unfused_maxpool, dim3(grid_for(planes * (H / 2) * (W / 2))), dim3(256), 0, stream, in,
                     in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, planes, H, W);
  return hipGetLastError();
}

hipError_t launch_unfused_channel_softmax(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t batch,
                                         int channels, int64_t spatial, hipStream_t stream) {
  hipLaunchKernelGGL(kf_unfused_channel_softmax, dim3(grid_for(batch * spatial)), dim3(256), 0, stream, in,
                     in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, batch, channels, spatial);
  return hipGetLastError();
}

hipError_t launch_unfused_maxpool3d(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int D,
                                    int H, int W, hipStream_t stream) {
  hipLaunchKernelGGL(kf_unfused_maxpool3d, dim3(grid_for(planes * (D / 2) * (H / 2) * (W / 2))), dim3(256), 0,
                     stream, in, in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, planes, D, H, W);
  return hipGetLastError();
}

}  // namespace kf
