// Row finishing kernels for row-wise softmax / logsumexp wider than a tile.
//
// The contraction kernel leaves, per (row m, 256-column tile t), the pair
// (mu_t, s_t) = (max over the tile of h, sum over the tile of e^(h - mu_t)).
// The row's statistics follow from the exact identities
//     mu = max_t mu_t,     S = sum_t s_t e^(mu_t - mu),
//     logsumexp = mu + ln S,
//     softmax_j = e^(h_j - mu_t) * e^(mu_t - mu) / S   for column j in tile t,
// which is the hierarchical, online form of softmax the paper's Appendix A
// (algorithmic optimisation: online softmax) and Appendix B (hierarchical
// reductions, normalise before exponentiating) recommend.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

// One row per group of L = 2^lanes_log2 lanes (the tile count rounded up to
// a power of two, at most 64): lane i of a group takes tiles i, i + L, ... of
// its row, so one load instruction of a wave covers 64 consecutive pairs, and
// the max and the sum are combined across the group by xor exchanges (every
// lane of the wave takes part in them, rows past M with nothing loaded).
__global__ __launch_bounds__(256) void kf_row_logsumexp_finish(const float2* __restrict__ part, int tiles,
                                                                int lanes_log2, int64_t M, float* __restrict__ out) {
  const int L = 1 << lanes_log2;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t m = gid >> lanes_log2;
  const int i = (int)(gid & (L - 1));
  const bool live = m < M;
  const float2* pr = part + m * tiles;
  float mu = -INFINITY;
  if (live)
    for (int t = i; t < tiles; t += L) mu = fmaxf(mu, pr[t].x);
  for (int d = 1; d < L; d <<= 1) mu = fmaxf(mu, __shfl_xor(mu, d, 64));
  float s = 0.0f;
  if (live)
    for (int t = i; t < tiles; t += L) s += pr[t].y * expf(pr[t].x - mu);
  for (int d = 1; d < L; d <<= 1) s += __shfl_xor(s, d, 64);
  if (live && i == 0) out[m] = mu + logf(s);
}

constexpr int kMaxFinishTiles = 1024;

// One workgroup per row: factors f_t = e^(mu_t - mu) / S, then every 16-byte
// chunk of the row is scaled by the factor of its tile.  The row is taken in
// passes of 4 chunks per thread (16 KiB per workgroup for bf16), all four
// loads issued before any store, so that each thread keeps several reads in
// flight: the kernel only moves data, and its speed is the number of bytes
// in flight per CU.
__global__ __launch_bounds__(256) void kf_row_softmax_rescale(const float2* __restrict__ part, int tiles,
                                                               int64_t N, void* out, int64_t ldo,
                                                               int out_bf16) {
  __shared__ float2 ps[kMaxFinishTiles];
  __shared__ float fac[kMaxFinishTiles];
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x;
  for (int t = tid; t < tiles; t += 256) ps[t] = part[m * tiles + t];
  __syncthreads();
  float mu = -INFINITY;
  for (int t = 0; t < tiles; ++t) mu = fmaxf(mu, ps[t].x);
  float s = 0.0f;
  for (int t = 0; t < tiles; ++t) s += ps[t].y * expf(ps[t].x - mu);
  const float inv = 1.0f / s;
  for (int t = tid; t < tiles; t += 256) fac[t] = expf(ps[t].x - mu) * inv;
  __syncthreads();
  constexpr int U = 4;
  if (out_bf16) {
    uint16_t* row = reinterpret_cast<uint16_t*>(out) + m * ldo;
    const int64_t chunks = N / 8;  // N % 8 == 0 for bf16 outputs
    for (int64_t c0 = 0; c0 < chunks; c0 += 256 * U) {
      u32x4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c < chunks) w[u] = *reinterpret_cast<const u32x4*>(row + c * 8);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c >= chunks) continue;
        const float f = fac[(c * 8) >> 8];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[u][e] = pack_bf16x2(bf16_lo(w[u][e]) * f, bf16_hi(w[u][e]) * f);
        *reinterpret_cast<u32x4*>(row + c * 8) = w[u];
      }
    }
  } else {
    float* row = reinterpret_cast<float*>(out) + m * ldo;
    const int64_t chunks = N / 4;  // N % 4 == 0 for fp32 outputs of the matrix-core GEMMs
    for (int64_t c0 = 0; c0 < chunks; c0 += 256 * U) {
      f32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c < chunks) v[u] = *reinterpret_cast<const f32x4*>(row + c * 4);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c < chunks) *reinterpret_cast<f32x4*>(row + c * 4) = v[u] * fac[(c * 4) >> 8];
      }
    }
  }
}

hipError_t launch_row_finish(bool softmax, const void* partials, int tiles, int64_t M, int64_t N, void* out,
                             int64_t ldo, bool out_bf16, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (softmax) {
    hipLaunchKernelGGL(kf_row_softmax_rescale, dim3((unsigned)M), dim3(256), 0, stream,
                       reinterpret_cast<const float2*>(partials), tiles, N, out, ldo, out_bf16 ? 1 : 0);
  } else {
    int lanes_log2 = 0;
    while ((1 << lanes_log2) < tiles && lanes_log2 < 6) ++lanes_log2;
    const int64_t threads = M << lanes_log2;
    hipLaunchKernelGGL(kf_row_logsumexp_finish, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                       reinterpret_cast<const float2*>(partials), tiles, lanes_log2, M, reinterpret_cast<float*>(out));
  }
  return hipGetLastError();
}

int row_finish_max_tiles() { return kMaxFinishTiles; }

}  // namespace kf
