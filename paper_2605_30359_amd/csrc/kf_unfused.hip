// The unfused comparator: one kernel per op, every intermediate stored to
// device memory (bf16, or fp32 for fp32 chains) -- the one-kernel-per-operator
// form that operator fusion removes (Appendix A, "Operator Fusion"; the
// paper's speedups are measured against such eager operator chains).  The
// contraction itself reuses the fused kernels with an empty op list.
//
// All kernels here are memory-bound, so each is laid out for HBM bandwidth:
// every lane moves whole 16-byte chunks (8 bf16 or 4 fp32 values), a wave's
// accesses are contiguous, each lane has several chunks in flight before it
// uses the first, grid-stride launches are sized to what the device holds at
// once, and results are written with streaming (nontemporal) stores.  The row reductions (GroupNorm, softmax, logsumexp) run
// on the row-wise kernels of kf_rowwise.hip; the kernels below cover the
// element-wise ops, the residual add, the pools and the channel softmax, and
// keep a scalar form for shapes the vector forms do not tile.
#include <algorithm>

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

// Row softmax / logsumexp / cross-entropy over N columns: one workgroup per row.
__global__ __launch_bounds__(256) void kf_unfused_rowop(const void* in, int in_bf16, void* out, int out_bf16,
                                                        int64_t N, int kind, const int32_t* targets) {
  const bool softmax = kind == KF_OP_ROW_SOFTMAX;
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
    if (threadIdx.x == 0) {
      float r = m + logf(s);
      if (kind == KF_OP_ROW_CROSS_ENTROPY) {
        const int32_t t = targets[row];
        r = (t >= 0 && t < N) ? r - load_elem(in, base + t, in_bf16) : __builtin_nanf("");
      }
      reinterpret_cast<float*>(out)[row] = r;
    }
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


// ------------------------------------------------------------ vector forms

// chunk c of a tensor = values [8c, 8c + 8)
template <bool BF16>
__device__ __forceinline__ void load8(const void* p, int64_t c, float (&x)[8]) {
  if constexpr (BF16) {
    const u32x4 w = reinterpret_cast<const u32x4*>(p)[c];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = bf16_lo(w[e]);
      x[2 * e + 1] = bf16_hi(w[e]);
    }
  } else {
    const f32x4* f = reinterpret_cast<const f32x4*>(p) + 2 * c;
    const f32x4 lo = f[0], hi = f[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = lo[e];
      x[4 + e] = hi[e];
    }
  }
}
template <bool BF16>
__device__ __forceinline__ void store8(void* p, int64_t c, const float (&x)[8]) {
  if constexpr (BF16) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
    store_nt(reinterpret_cast<u32x4*>(p) + c, w);
  } else {
    f32x4* f = reinterpret_cast<f32x4*>(p) + 2 * c;
    store_nt(f, f32x4{x[0], x[1], x[2], x[3]});
    store_nt(f + 1, f32x4{x[4], x[5], x[6], x[7]});
  }
}

enum VecMode { kVecOp = 0, kVecBiasCols = 1, kVecBiasPlane = 2, kVecResidual = 3 };
constexpr int kVecUnroll = 1;  // chunks per lane and iteration (1 ran faster than 2 or 4: more waves)

// out = op(in) over `chunks` chunks: an element-wise op, + bias per column of
// rows of fmod values (kVecBiasCols, fmod % 8 == 0), + bias per plane of
// plane_chunks chunks (kVecBiasPlane, channel = plane % fmod), or +
// residual.  Each lane loads kVecUnroll chunks (a grid stride apart, so each
// load instruction of a wave is contiguous) before it computes.
template <bool IN_BF16, bool OUT_BF16, bool RES_BF16, int MODE>
__global__ __launch_bounds__(256) void kf_unfused_vec(const void* in, void* out, int64_t chunks, int kind, float p0,
                                                      float p1, const float* bias, const void* res,
                                                      int64_t plane_chunks, int64_t fmod) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t c0 = (int64_t)blockIdx.x * 256 + threadIdx.x; c0 < chunks; c0 += stride * kVecUnroll) {
    float x[kVecUnroll][8], r[kVecUnroll][8];
#pragma unroll
    for (int u = 0; u < kVecUnroll; ++u) {
      const int64_t c = c0 + u * stride;
      if (c < chunks) {
        load8<IN_BF16>(in, c, x[u]);
        if constexpr (MODE == kVecResidual) load8<RES_BF16>(res, c, r[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < kVecUnroll; ++u) {
      const int64_t c = c0 + u * stride;
      if (c >= chunks) continue;
      if constexpr (MODE == kVecOp) {
        apply_elementwise_array<8>(kind, p0, p1, x[u]);
      } else if constexpr (MODE == kVecBiasCols) {
        const f32x4* b = reinterpret_cast<const f32x4*>(bias + (c * 8) % fmod);
        const f32x4 lo = b[0], hi = b[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[u][e] += lo[e];
          x[u][4 + e] += hi[e];
        }
      } else if constexpr (MODE == kVecBiasPlane) {
        const float b = bias[(c / plane_chunks) % fmod];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[u][e] += b;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[u][e] += r[u][e];
      }
      store8<OUT_BF16>(out, c, x[u]);
    }
  }
}

// MaxPool2d(2, 2) of bf16 [planes][H][W] with W % 16 == 0: each lane takes 16
// columns of a row pair (four 16-byte loads) and writes 8 outputs (one
// 16-byte store).
__global__ __launch_bounds__(256) void kf_unfused_maxpool_vec(const uint16_t* in, uint16_t* out, int64_t planes,
                                                              int H, int W) {
  const int Ho = H / 2, Wv = W / 16;  // output chunks per output row
  const int64_t n = planes * Ho * Wv;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    const int64_t pr = i / Wv;  // plane * Ho + output row
    const int q = (int)(i % Wv);
    const int64_t pl = pr / Ho;
    const int ph = (int)(pr % Ho);
    const u32x4* r0 = reinterpret_cast<const u32x4*>(in + (pl * H + 2 * ph) * (int64_t)W + 16 * q);
    const u32x4* r1 = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(r0) + W);
    const u32x4 a0 = r0[0], a1 = r0[1], b0 = r1[0], b1 = r1[1];
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t wa = e < 2 ? a0[2 * e] : a1[2 * e - 4], wb = e < 2 ? a0[2 * e + 1] : a1[2 * e - 3];
      const uint32_t va = e < 2 ? b0[2 * e] : b1[2 * e - 4], vb = e < 2 ? b0[2 * e + 1] : b1[2 * e - 3];
      const float m0 = fmaxf(fmaxf(bf16_lo(wa), bf16_hi(wa)), fmaxf(bf16_lo(va), bf16_hi(va)));
      const float m1 = fmaxf(fmaxf(bf16_lo(wb), bf16_hi(wb)), fmaxf(bf16_lo(vb), bf16_hi(vb)));
      // a maximum of bf16 values is one of them: the packing is exact
      o[e] = pack_bf16x2(m0, m1);
    }
    store_nt(reinterpret_cast<u32x4*>(out) + i, o);
  }
}

// MaxPool3d(2) of bf16 [planes][D][H][W] with W % 16 == 0, floor mode: each
// lane takes 16 columns of the 2 x 2 rows of one output row (eight 16-byte
// loads) and writes 8 outputs.
__global__ __launch_bounds__(256) void kf_unfused_maxpool3d_vec(const uint16_t* in, uint16_t* out, int64_t planes,
                                                                int D, int H, int W) {
  const int Do = D / 2, Ho = H / 2, Wv = W / 16;
  const int64_t n = planes * Do * Ho * Wv;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    const int q = (int)(i % Wv);
    const int64_t r = i / Wv;
    const int ph = (int)(r % Ho);
    const int64_t r2 = r / Ho;
    const int pd = (int)(r2 % Do);
    const int64_t pl = r2 / Do;
    float m[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
#pragma unroll
    for (int dd = 0; dd < 2; ++dd)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const u32x4* row =
            reinterpret_cast<const u32x4*>(in + ((pl * D + 2 * pd + dd) * H + 2 * ph + hh) * (int64_t)W + 16 * q);
        const u32x4 lo = row[0], hi = row[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          m[e] = fmaxf(m[e], fmaxf(bf16_lo(lo[e]), bf16_hi(lo[e])));
          m[4 + e] = fmaxf(m[4 + e], fmaxf(bf16_lo(hi[e]), bf16_hi(hi[e])));
        }
      }
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(m[2 * e], m[2 * e + 1]);
    store_nt(reinterpret_cast<u32x4*>(out) + i, o);
  }
}

// Softmax over the C = 64 channels of bf16 [batch][64][S] with S % 2 == 0:
// each lane takes 2 consecutive positions and holds all 64 channels of them
// in registers (64 4-byte loads, one per channel plane; a wave's load covers
// 256 contiguous bytes), so the input is read once: max, then the sum of
// e^(h - max), then the normalised store.
constexpr int kCsmChannels = 64;
__global__ __launch_bounds__(256) void kf_unfused_channel_softmax_vec(const uint16_t* in, uint16_t* out,
                                                                      int64_t batch, int64_t S) {
  const int64_t per = S / 2;
  const int64_t n = batch * per;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    const int64_t base = (i / per) * kCsmChannels * S + (i % per) * 2;
    uint32_t v[kCsmChannels];
#pragma unroll
    for (int c = 0; c < kCsmChannels; ++c) v[c] = *reinterpret_cast<const uint32_t*>(in + base + c * S);
    float m0 = -INFINITY, m1 = -INFINITY;
#pragma unroll
    for (int c = 0; c < kCsmChannels; ++c) {
      m0 = fmaxf(m0, bf16_lo(v[c]));
      m1 = fmaxf(m1, bf16_hi(v[c]));
    }
    const float l0 = m0 * kLog2e, l1 = m1 * kLog2e;
    float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
    for (int c = 0; c < kCsmChannels; ++c) {
      s0 += __builtin_amdgcn_exp2f(fmaf(bf16_lo(v[c]), kLog2e, -l0));
      s1 += __builtin_amdgcn_exp2f(fmaf(bf16_hi(v[c]), kLog2e, -l1));
    }
    const float i0 = 1.0f / s0, i1 = 1.0f / s1;
#pragma unroll
    for (int c = 0; c < kCsmChannels; ++c)
      store_nt(reinterpret_cast<uint32_t*>(out + base + c * S),
               pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(bf16_lo(v[c]), kLog2e, -l0)) * i0,
                           __builtin_amdgcn_exp2f(fmaf(bf16_hi(v[c]), kLog2e, -l1)) * i1));
  }
}

static unsigned grid_for(int64_t n) {
  const int64_t g = (n + 255) / 256;
  return (unsigned)(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

// workgroups of a grid-stride launch over n items at `per_lane` items per
// lane and iteration: enough for one iteration each, at most what the device
// holds at once
static unsigned stream_grid(int64_t n, int per_lane, int resident) {
  const int64_t g = (n + 256 * per_lane - 1) / (256 * per_lane);
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(g, resident));
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <int MODE, bool RES_BF16>
static void launch_vec(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t chunks, int kind, float p0,
                       float p1, const float* bias, const void* res, int64_t plane_chunks, int64_t fmod,
                       hipStream_t stream) {
#define KF_VEC_LAUNCH(IB, OB)                                                                                   \
  do {                                                                                                          \
    static const int resident = resident_blocks(kf_unfused_vec<IB, OB, RES_BF16, MODE>, 256);                   \
    hipLaunchKernelGGL((kf_unfused_vec<IB, OB, RES_BF16, MODE>), dim3(stream_grid(chunks, kVecUnroll, resident)), \
                       dim3(256), 0, stream, in, out, chunks, kind, p0, p1, bias, res, plane_chunks, fmod);      \
  } while (0)
  if (in_bf16 && out_bf16)
    KF_VEC_LAUNCH(true, true);
  else if (in_bf16)
    KF_VEC_LAUNCH(true, false);
  else if (out_bf16)
    KF_VEC_LAUNCH(false, true);
  else
    KF_VEC_LAUNCH(false, false);
#undef KF_VEC_LAUNCH
}

hipError_t launch_unfused_elementwise(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t n, int kind,
                                      float p0, float p1, const float* bias, int64_t fdiv, int64_t fmod,
                                      hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const bool vec = (n & 7) == 0 && aligned16(in) && aligned16(out);
  if (vec && kind != KF_OP_BIAS) {
    launch_vec<kVecOp, true>(in, in_bf16, out, out_bf16, n / 8, kind, p0, p1, nullptr, nullptr, 1, 1, stream);
    return hipGetLastError();
  }
  if (vec && kind == KF_OP_BIAS && fdiv == 1 && fmod % 8 == 0 && aligned16(bias)) {
    launch_vec<kVecBiasCols, true>(in, in_bf16, out, out_bf16, n / 8, kind, p0, p1, bias, nullptr, 1, fmod, stream);
    return hipGetLastError();
  }
  if (vec && kind == KF_OP_BIAS && fdiv % 8 == 0) {
    launch_vec<kVecBiasPlane, true>(in, in_bf16, out, out_bf16, n / 8, kind, p0, p1, bias, nullptr, fdiv / 8, fmod,
                                    stream);
    return hipGetLastError();
  }
  const int64_t work = (in_bf16 && out_bf16 && (n & 7) == 0) ? n / 8 : n;
  hipLaunchKernelGGL(kf_unfused_elementwise, dim3(grid_for(work)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, n, kind, p0, p1, bias, fdiv, fmod);
  return hipGetLastError();
}

hipError_t launch_unfused_residual(const void* in, bool in_bf16, const void* res, bool res_bf16, void* out,
                                   bool out_bf16, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if ((n & 7) == 0 && aligned16(in) && aligned16(out) && aligned16(res)) {
    if (res_bf16)
      launch_vec<kVecResidual, true>(in, in_bf16, out, out_bf16, n / 8, 0, 0.f, 0.f, nullptr, res, 1, 1, stream);
    else
      launch_vec<kVecResidual, false>(in, in_bf16, out, out_bf16, n / 8, 0, 0.f, 0.f, nullptr, res, 1, 1, stream);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(kf_unfused_residual, dim3(grid_for(n)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, res,
                     res_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, n);
  return hipGetLastError();
}

hipError_t launch_unfused_groupnorm(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                    int groups, float eps, const float* gamma, const float* beta,
                                    hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const int64_t gw = N / groups;
  if (N % 8 == 0 && gw % 8 == 0 && N <= rowwise_max_cols() && aligned16(in) && aligned16(out) && aligned16(gamma) &&
      aligned16(beta)) {
    RowArgs r{};
    r.a = in;
    r.M = rows;
    r.N = N;
    r.lda = N;
    r.in_bf16 = in_bf16;
    r.prog.n = 1;
    r.prog.op[0] = EpiOp{KF_OP_GROUPNORM, groups, eps, 0.0f};
    r.gamma = gamma;
    r.beta = beta;
    r.out = out;
    r.ldo = N;
    r.out_bf16 = out_bf16;
    r.gn_group = (int32_t)gw;
    return launch_rowwise(r, kChainGroupNorm, stream);
  }
  hipLaunchKernelGGL(kf_unfused_groupnorm, dim3((unsigned)(rows * groups)), dim3(256), 0, stream, in,
                     in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, N, (int)gw, eps, gamma, beta);
  return hipGetLastError();
}

hipError_t launch_unfused_rowop(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t rows, int64_t N,
                                int kind, const int32_t* targets, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const bool softmax = kind == KF_OP_ROW_SOFTMAX;
  if (N % 8 == 0 && (N <= rowwise_max_cols() || !softmax) && aligned16(in) && (!softmax || aligned16(out))) {
    RowArgs r{};
    r.a = in;
    r.M = rows;
    r.N = N;
    r.lda = N;
    r.in_bf16 = in_bf16;
    r.prog.n = 1;
    r.prog.op[0] = EpiOp{kind, 0, 0.0f, 0.0f};
    r.out = out;
    r.ldo = softmax ? N : 1;
    r.out_bf16 = softmax && out_bf16;
    r.targets = targets;
    return launch_rowwise(r,
                          softmax                           ? kChainRowSoftmax
                          : kind == KF_OP_ROW_LOGSUMEXP     ? kChainRowLogsumexp
                                                            : kChainRowCrossEntropy,
                          stream);
  }
  hipLaunchKernelGGL(kf_unfused_rowop, dim3((unsigned)rows), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, N, kind, targets);
  return hipGetLastError();
}

hipError_t launch_unfused_maxpool(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int H,
                                  int W, hipStream_t stream) {
  const int64_t n = planes * (H / 2) * (W / 2);
  if (n <= 0) return hipSuccess;
  if (in_bf16 && out_bf16 && W % 16 == 0 && aligned16(in) && aligned16(out)) {
    static const int resident = resident_blocks(kf_unfused_maxpool_vec, 256);
    hipLaunchKernelGGL(kf_unfused_maxpool_vec, dim3(stream_grid(n / 8, 1, resident)), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(in), static_cast<uint16_t*>(out), planes, H, W);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(kf_unfused_maxpool, dim3(grid_for(n)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, planes, H, W);
  return hipGetLastError();
}

hipError_t launch_unfused_channel_softmax(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t batch,
                                         int channels, int64_t spatial, hipStream_t stream) {
  if (batch * spatial <= 0) return hipSuccess;
  if (in_bf16 && out_bf16 && channels == kCsmChannels && spatial % 2 == 0 &&
      (reinterpret_cast<uintptr_t>(in) & 3) == 0 && (reinterpret_cast<uintptr_t>(out) & 3) == 0) {
    static const int resident = resident_blocks(kf_unfused_channel_softmax_vec, 256);
    hipLaunchKernelGGL(kf_unfused_channel_softmax_vec, dim3(stream_grid(batch * spatial / 2, 1, resident)), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(in), static_cast<uint16_t*>(out), batch, spatial);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(kf_unfused_channel_softmax, dim3(grid_for(batch * spatial)), dim3(256), 0, stream, in,
                     in_bf16 ? 1 : 0, out, out_bf16 ? 1 : 0, batch, channels, spatial);
  return hipGetLastError();
}

hipError_t launch_unfused_maxpool3d(const void* in, bool in_bf16, void* out, bool out_bf16, int64_t planes, int D,
                                    int H, int W, hipStream_t stream) {
  const int64_t n = planes * (D / 2) * (H / 2) * (W / 2);
  if (n <= 0) return hipSuccess;
  if (in_bf16 && out_bf16 && W % 16 == 0 && aligned16(in) && aligned16(out)) {
    static const int resident = resident_blocks(kf_unfused_maxpool3d_vec, 256);
    hipLaunchKernelGGL(kf_unfused_maxpool3d_vec, dim3(stream_grid(n / 8, 1, resident)), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(in), static_cast<uint16_t*>(out), planes, D, H, W);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(kf_unfused_maxpool3d, dim3(grid_for(n)), dim3(256), 0, stream, in, in_bf16 ? 1 : 0, out,
                     out_bf16 ? 1 : 0, planes, D, H, W);
  return hipGetLastError();
}

}  // namespace kf
