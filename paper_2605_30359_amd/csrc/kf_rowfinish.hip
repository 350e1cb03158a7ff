// Row finishing kernels for row-wise softmax / logsumexp wider than a tile.
//
// The contraction kernel leaves, per (row m, 256-column tile t), the pair
// (mu_t, s_t) = (max over the tile of h, sum over the tile of e^(h - mu_t)).
// The row's statistics follow from the exact identities
//     mu = max_t mu_t,     S = sum_t s_t e^(mu_t - mu),
//     logsumexp = mu + ln S,
//     softmax_j = e^(h_j - mu_t) * e^(mu_t - mu) / S   for column j in tile t,
//     cross-entropy = logsumexp - h_target  (h_target left by the tile holding it),
// which is the hierarchical, online form of softmax the paper's Appendix A
// (algorithmic optimisation: online softmax) and Appendix B (hierarchical
// reductions, normalise before exponentiating) recommend.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

// One row per group of L = 2^lanes_log2 lanes (the tile count rounded up to
// a power of two, at most 64): lane i of a group takes tiles i, i + L, ... of
// its row, so one load instruction of a wave covers 64 consecutive pairs
// when the tile count is a power of two (and nearly so otherwise), and
// the max and the sum are combined across the group by xor exchanges (every
// lane of the wave takes part in them, rows past M with nothing loaded).
__global__ __launch_bounds__(256) void kf_row_logsumexp_finish(const float2* __restrict__ part, int tiles,
                                                                int lanes_log2, int64_t M, float* __restrict__ out,
                                                                const int32_t* __restrict__ targets,
                                                                const float* __restrict__ tlogit, int64_t N) {
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
  if (live && i == 0) {
    float r = mu + logf(s);
    if (targets) {
      const int32_t t = targets[m];
      r = (t >= 0 && t < N) ? r - tlogit[m] : __builtin_nanf("");
    }
    out[m] = r;
  }
}

constexpr int kMaxFinishTiles = 1024;

// One workgroup per row: factors f_t = e^(mu_t - mu) / S, then every 16-byte
// chunk of the row is scaled by the factor of its tile.  The row is taken in
// passes of 4 chunks per thread (16 KiB per workgroup for bf16), all four
// loads issued before any store, so that each thread keeps several reads in
// flight: the kernel only moves data, and its speed is the number of bytes
// in flight per CU.  The first pass's loads do not depend on the factors and
// go out before the partials are read, so the two memory latencies overlap.
// mu and S are combined by every wave over the tiles in lane order (lane i
// takes tiles i, i + 64, ...), then across the wave by xor exchanges.
template <typename V, int U>
__device__ __forceinline__ void load_pass(const V* row, int64_t chunks, int64_t c0, int tid, V (&w)[U]) {
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t c = c0 + u * 256 + tid;
    if (c < chunks) w[u] = row[c];
  }
}

__global__ __launch_bounds__(256) void kf_row_softmax_rescale(const float2* __restrict__ part, int tiles,
                                                               int64_t N, void* out, int64_t ldo,
                                                               int out_bf16) {
  __shared__ float fac[kMaxFinishTiles];
  constexpr int U = 4;
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const bool bf = out_bf16 != 0;
  u32x4* rowb = reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(out) + m * ldo);
  f32x4* rowf = reinterpret_cast<f32x4*>(reinterpret_cast<float*>(out) + m * ldo);
  // N % 8 == 0 for bf16 outputs, N % 4 == 0 for fp32 outputs of the matrix-core GEMMs
  const int64_t chunks = bf ? N / 8 : N / 4;
  const int shift = bf ? 5 : 6;  // chunk -> 256-column tile
  u32x4 w[U];
  f32x4 v[U];
  if (bf)
    load_pass(rowb, chunks, 0, tid, w);
  else
    load_pass(rowf, chunks, 0, tid, v);

  const float2* pr = part + m * tiles;
  float mu = -INFINITY;
  for (int t = lane; t < tiles; t += 64) mu = fmaxf(mu, pr[t].x);
  for (int d = 1; d < 64; d <<= 1) mu = fmaxf(mu, __shfl_xor(mu, d, 64));
  float s = 0.0f;
  for (int t = lane; t < tiles; t += 64) s += pr[t].y * expf(pr[t].x - mu);
  for (int d = 1; d < 64; d <<= 1) s += __shfl_xor(s, d, 64);
  const float inv = 1.0f / s;
  for (int t = tid; t < tiles; t += 256) fac[t] = expf(pr[t].x - mu) * inv;
  __syncthreads();

  for (int64_t c0 = 0; c0 < chunks; c0 += 256 * U) {
    if (bf) {
      if (c0 > 0) load_pass(rowb, chunks, c0, tid, w);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c >= chunks) continue;
        const float f = fac[c >> shift];
#pragma unroll
        for (int e = 0; e < 4; ++e) w[u][e] = pack_bf16x2(bf16_lo(w[u][e]) * f, bf16_hi(w[u][e]) * f);
        store_nt(rowb + c, w[u]);
      }
    } else {
      if (c0 > 0) load_pass(rowf, chunks, c0, tid, v);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t c = c0 + u * 256 + tid;
        if (c < chunks) store_nt(rowf + c, v[u] * fac[c >> shift]);
      }
    }
  }
}

hipError_t launch_row_finish(bool softmax, const void* partials, int tiles, int64_t M, int64_t N, void* out,
                             int64_t ldo, bool out_bf16, hipStream_t stream, const int32_t* targets,
                             const float* tlogit) {
  if (M <= 0) return hipSuccess;
  if (softmax) {
    hipLaunchKernelGGL(kf_row_softmax_rescale, dim3((unsigned)M), dim3(256), 0, stream,
                       reinterpret_cast<const float2*>(partials), tiles, N, out, ldo, out_bf16 ? 1 : 0);
  } else {
    int lanes_log2 = 0;
    while ((1 << lanes_log2) < tiles && lanes_log2 < 6) ++lanes_log2;
    const int64_t threads = M << lanes_log2;
    hipLaunchKernelGGL(kf_row_logsumexp_finish, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                       reinterpret_cast<const float2*>(partials), tiles, lanes_log2, M, reinterpret_cast<float*>(out),
                       targets, tlogit, N);
  }
  return hipGetLastError();
}

int row_finish_max_tiles() { return kMaxFinishTiles; }

}  // namespace kf
