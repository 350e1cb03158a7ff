// The matrix cores' sustained rate with no memory traffic: a measured
// ceiling for the roofline beside the datasheet one.  The datasheet's dense
// peaks assume the 2.4 GHz peak engine clock; under sustained matrix-core
// load the clock is whatever power management allows, and this kernel
// reports both the rate and that clock.
//
// One workgroup of 4 waves per compute unit (its LDS allocation keeps a
// second one off the CU), so each SIMD runs one wave, which issues rounds of
// 8 independent 32x32 MFMAs from registers: the dependent chains are 8 long,
// so every MFMA can issue as soon as the pipe takes it.  The A operands
// rotate over 4 register sets and the B operands over 2, so consecutive
// MFMAs see different data, as in a GEMM (the power drawn, and with it the
// clock, depends on the operand bits changing).  Each workgroup stamps the
// shader-clock counter and the constant-rate counter at its start and end.
// Beside it, a plain device copy gives the memory side's measured ceiling.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeLds = 96 * 1024;  // more than half the CU's LDS: one workgroup per CU

// Lane-dependent operand bits (an integer hash of lane and register
// index): random signs and mantissas with a fixed small exponent -- e4m3
// bytes +-(1 .. 1.875) x 2^-3 (exponent field 4), bf16 half-words
// +-(1 .. 2) x 2^-5 (exponent field 122) -- so that the sums stay finite
// over any run.
__device__ __forceinline__ uint32_t probe_bits(uint32_t lane, uint32_t j, bool fp8) {
  uint32_t h = (lane * 0x9E3779B1u) ^ (j * 0x85EBCA77u);
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  return fp8 ? (h & 0x87878787u) | 0x20202020u : (h & 0x807F807Fu) | 0x3D003D00u;
}

}  // namespace

template <bool FP8>
__global__ __launch_bounds__(kProbeThreads, 1) void kf_mfma_probe(int64_t iters, float* __restrict__ sink,
                                                                  long long* __restrict__ stamps) {
  __shared__ float pad[kProbeLds / 4];
  const long long c0 = clock64(), w0 = wall_clock64();
  const uint32_t lane = threadIdx.x & 63;
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[j][i] = 0.0f;

  if constexpr (FP8) {
    i32x8 a[4], b[2];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) a[j][e] = (int)probe_bits(lane, 8 * j + e, true);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) b[j][e] = (int)probe_bits(lane, 100 + 8 * j + e, true);
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[j & 3], b[j >> 2], acc[j], 0, 0, 0, 127, 0, 127);
    }
  } else {
    u32x4 a[4], b[2];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) a[j][e] = probe_bits(lane, 4 * j + e, false);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) b[j][e] = probe_bits(lane, 100 + 4 * j + e, false);
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[j & 3]),
                                                         __builtin_bit_cast(bf16x8, b[j >> 2]), acc[j], 0, 0, 0);
    }
  }

  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[j][i];
  if (iters < 0) pad[threadIdx.x] = s;  // never taken: keeps the LDS allocation
  sink[(int64_t)blockIdx.x * kProbeThreads + threadIdx.x] = s;
  const long long c1 = clock64(), w1 = wall_clock64();
  if (threadIdx.x == 0) {
    long long* st = stamps + 4 * (int64_t)blockIdx.x;
    st[0] = c0;
    st[1] = c1;
    st[2] = w0;
    st[3] = w1;
  }
}

// A plain device copy of n 16-byte chunks: the memory side's measured
// ceiling.  Spans of 256 x kCopyUnroll chunks per workgroup; each lane issues its kCopyUnroll loads (256 chunks apart, so
// every load instruction of a wave reads 1 KiB of contiguous memory) before
// its stores, which are streaming stores as in the library's memory-bound
// kernels.
constexpr int kCopyUnroll = 8;
__global__ __launch_bounds__(256) void kf_copy_probe(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                     int64_t n) {
  constexpr int64_t span = 256 * kCopyUnroll;
  for (int64_t b0 = (int64_t)blockIdx.x * span; b0 < n; b0 += (int64_t)gridDim.x * span) {
    u32x4 v[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int64_t c = b0 + u * 256 + threadIdx.x;
      if (c < n) v[u] = src[c];
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int64_t c = b0 + u * 256 + threadIdx.x;
      if (c < n) store_nt(dst + c, v[u]);
    }
  }
}

int probe_threads() { return kProbeThreads; }

hipError_t launch_copy_probe(const void* src, void* dst, int64_t chunks, hipStream_t stream) {
  // one span per workgroup (at 2 x 512 MiB this measured 1-2% above a
  // resident-sized grid that loops); the loop covers grids capped at 2^31
  const int64_t need = (chunks + 256 * kCopyUnroll - 1) / (256 * kCopyUnroll);
  hipLaunchKernelGGL(kf_copy_probe, dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, INT32_MAX))),
                     dim3(256), 0, stream, static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), chunks);
  return hipGetLastError();
}

hipError_t launch_mfma_probe(bool fp8, int64_t iters, int workgroups, float* sink, long long* stamps,
                             hipStream_t stream) {
  if (fp8)
    hipLaunchKernelGGL(kf_mfma_probe<true>, dim3((unsigned)workgroups), dim3(kProbeThreads), 0, stream, iters, sink,
                       stamps);
  else
    hipLaunchKernelGGL(kf_mfma_probe<false>, dim3((unsigned)workgroups), dim3(kProbeThreads), 0, stream, iters, sink,
                       stamps);
  return hipGetLastError();
}

}  // namespace kf
