// The general 3x3x3 convolution (PyTorch Conv3d: stride 1, no padding, no
// dilation, groups 1) with a fused bias and element-wise ops, for every shape
// and input layout the tiled Conv3d kernel does not take: any batch, cin,
// cout and D, H, W >= 3, the input addressed through its element strides
// (contiguous NCDHW or channels-last), the output NCDHW.
//
// Implicit GEMM: m = output position, n = output channel, k = (chunk of 16
// input channels, kd, kh, kw).  Tile: 4 output rows x 32 columns at one output
// depth x 128 output channels per workgroup of 4 waves; wave w owns channels
// [32 w, 32 w + 32) and all four rows (four 32 x 32 MFMA blocks, so each
// weight fragment serves four).  For each (chunk, kd) the 6 x 34 x 16 input
// patch at depth od + kd (zero past the volume and past cin) is staged in LDS
// as [pixel][16 channels] -- an A fragment is one 16-byte read -- loaded into
// registers one step ahead; the 9 (kh, kw) taps read it at shifted pixels.
// The B fragments come from the weights repacked to [tap][cout][cin rounded
// up to 16] (zero-padded) straight from global memory, where they stay in L2.
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int kG3Cols = 32, kG3Rows = 4, kG3Co = 128;
constexpr int kG3PatchCols = kG3Cols + 2, kG3PatchRows = kG3Rows + 2;
constexpr int kG3Patch = 16 * kG3PatchRows * kG3PatchCols;  // 3264 elements per step
constexpr int kG3Loads = (kG3Patch + 255) / 256;           // 13 per thread

__host__ __device__ int g3_cin_pad(int cin) { return (cin + 15) / 16 * 16; }

}  // namespace

// wp[tap][co][ci] = w[co][ci][kd][kh][kw] (tap = 9 kd + 3 kh + kw) for
// ci < cin, 0 up to the padded cin
__global__ __launch_bounds__(256) void kf_conv3d_pack_weights_gen(const uint16_t* __restrict__ w,
                                                                  uint16_t* __restrict__ wp, int cout, int cin,
                                                                  int cin16) {
  const int64_t pairs = (int64_t)cout * cin16;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < pairs; e += (int64_t)gridDim.x * 256) {
    const int co = (int)(e / cin16), ci = (int)(e % cin16);
    for (int tap = 0; tap < 27; ++tap)
      wp[tap * pairs + e] = ci < cin ? w[((int64_t)co * cin + ci) * 27 + tap] : (uint16_t)0;
  }
}

__global__ __launch_bounds__(256) void kf_conv3d_bf16_gen(Conv3dGenArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(16))) uint16_t sP[kG3Patch];  // [row][col][16 ci]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int D = p.D, H = p.H, W = p.W, cin = p.cin, cout = p.cout;
  const int Do = D - 2, Ho = H - 2, Wo = W - 2;
  const int cin16 = g3_cin_pad(cin);
  const int chunks = cin16 / 16;
  const int tiles_co = (cout + kG3Co - 1) / kG3Co;
  const int tiles_w = (Wo + kG3Cols - 1) / kG3Cols;
  const int tiles_h = (Ho + kG3Rows - 1) / kG3Rows;
  int64_t b = blockIdx.x;
  const int tc = (int)(b % tiles_co);
  b /= tiles_co;
  const int tw = (int)(b % tiles_w);
  b /= tiles_w;
  const int th = (int)(b % tiles_h);
  b /= tiles_h;
  const int od = (int)(b % Do);
  const int64_t n = b / Do;
  const int oh0 = th * kG3Rows, ow0 = tw * kG3Cols;
  const int co0 = tc * kG3Co + wave * 32;
  const bool wave_live = co0 < cout;  // waves past cout compute nothing (they still meet every barrier)
  const uint16_t* x = reinterpret_cast<const uint16_t*>(p.x) + n * p.sn;

  // this thread's patch elements: e = tid + 256 j -> (ci, row, col), ci fastest
  uint16_t pre[kG3Loads];
  auto load_step = [&](int s) {  // step s = (chunk s / 3, kd s % 3)
    const int c = s / 3, kd = s - 3 * c;
#pragma unroll
    for (int j = 0; j < kG3Loads; ++j) {
      const int e = tid + 256 * j;
      const int ci = e & 15, pix = e >> 4;
      const int row = pix / kG3PatchCols, col = pix - row * kG3PatchCols;
      const int ih = oh0 + row, iw = ow0 + col, cc = c * 16 + ci;
      pre[j] = (e < kG3Patch && cc < cin && ih < H && iw < W)
                   ? x[cc * p.sc + (int64_t)(od + kd) * p.sd + (int64_t)ih * p.sh + (int64_t)iw * p.sw]
                   : (uint16_t)0;
    }
  };
  auto store_step = [&]() {
#pragma unroll
    for (int j = 0; j < kG3Loads; ++j) {
      const int e = tid + 256 * j;
      if (e < kG3Patch) sP[e] = pre[j];
    }
  };
  // B fragments of a step: lane (co0 + lane % 32, channels 8 (lane / 32) .. + 7)
  const int r32 = lane & 31, kg = lane >> 5;
  const int co_l = co0 + r32;
  const int64_t taps_stride = (int64_t)cout * cin16;
  u32x4 fb[9];
  auto load_b = [&](int s) {
    const int c = s / 3, kd = s - 3 * c;
#pragma unroll
    for (int t = 0; t < 9; ++t)
      fb[t] = co_l < cout ? *reinterpret_cast<const u32x4*>(wp + (kd * 9 + t) * taps_stride + (int64_t)co_l * cin16 +
                                                           c * 16 + kg * 8)
                          : u32x4{0u, 0u, 0u, 0u};
  };

  f32x16 acc[kG3Rows];
#pragma unroll
  for (int r = 0; r < kG3Rows; ++r)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[r][i] = 0.0f;

  const int steps = chunks * 3;
  load_step(0);
  store_step();
  __syncthreads();
  for (int s = 0; s < steps; ++s) {
    if (wave_live) load_b(s);
    if (s + 1 < steps) load_step(s + 1);
    if (wave_live) {
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int kh = t / 3, kw = t % 3;
#pragma unroll
        for (int r = 0; r < kG3Rows; ++r) {
          const int pix = (r + kh) * kG3PatchCols + r32 + kw;
          const u32x4 a = *reinterpret_cast<const u32x4*>(sP + pix * 16 + kg * 8);
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                           __builtin_bit_cast(bf16x8, fb[t]), acc[r], 0, 0, 0);
        }
      }
    }
    __syncthreads();
    if (s + 1 < steps) {
      store_step();
      __syncthreads();
    }
  }
  if (!wave_live || co_l >= cout) return;

  // epilogue: acc[r][i] = output row oh0 + r, column ow0 + (i / 4) * 8 +
  // (lane / 32) * 4 + i % 4, channel co_l; the op list in order (bias and
  // element-wise ops only)
  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const float bias = p.bias ? p.bias[co_l] : 0.0f;
  uint16_t* out = reinterpret_cast<uint16_t*>(p.out) + (((n * cout + co_l) * Do + od) * Ho) * (int64_t)Wo;
#pragma unroll
  for (int r = 0; r < kG3Rows; ++r) {
    float v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = acc[r][i];
    for (int o = 0; o < nops; ++o) {
      const int kind = op_kind(ops, o);
      if (kind == KF_OP_BIAS) {
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] += bias;
      } else {
        apply_elementwise_array<16>(kind, op_p0(ops, o), op_p1(ops, o), v);
      }
    }
    const int oh = oh0 + r;
    if (oh >= Ho) continue;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int ow = ow0 + (i / 4) * 8 + kg * 4 + (i & 3);
      if (ow < Wo) out[(int64_t)oh * Wo + ow] = (uint16_t)f32_to_bf16_rne(v[i]);
    }
  }
}

int64_t conv3d_gen_tiles(int64_t batch, int64_t D, int64_t H, int64_t W, int64_t cout) {
  return batch * (D - 2) * ((H - 2 + kG3Rows - 1) / kG3Rows) * ((W - 2 + kG3Cols - 1) / kG3Cols) *
         ((cout + kG3Co - 1) / kG3Co);
}

size_t conv3d_gen_packed_bytes(int64_t cout, int64_t cin) { return (size_t)27 * cout * g3_cin_pad((int)cin) * 2; }

hipError_t launch_conv3d_gen_pack(const void* w, void* packed, int cout, int cin, hipStream_t stream) {
  const int cin16 = g3_cin_pad(cin);
  const int64_t pairs = (int64_t)cout * cin16;
  const unsigned grid = (unsigned)std::min<int64_t>((pairs + 255) / 256, 4096);
  hipLaunchKernelGGL(kf_conv3d_pack_weights_gen, dim3(grid > 0 ? grid : 1), dim3(256), 0, stream,
                     reinterpret_cast<const uint16_t*>(w), reinterpret_cast<uint16_t*>(packed), cout, cin, cin16);
  return hipGetLastError();
}

hipError_t launch_conv3d_gen(const Conv3dGenArgs& args, const void* packed, hipStream_t stream) {
  const int64_t tiles = conv3d_gen_tiles(args.batch, args.D, args.H, args.W, args.cout);
  if (tiles <= 0) return hipSuccess;
  if (tiles > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kf_conv3d_bf16_gen, dim3((unsigned)tiles), dim3(256), 0, stream, args,
                     reinterpret_cast<const uint16_t*>(packed));
  return hipGetLastError();
}

}  // namespace kf
