// 3x3 convolution (stride 1, zero padding 1, NCHW / OIHW, bf16) as an
// implicit GEMM on the matrix cores, with the element-wise ops and the 2x2
// max-pool of the op list fused into the epilogue.  This is the paper's
// conv-centred fused operator family (Evaluation, Table 2: conv-centred
// chains; Appendix C: a convolution followed by pooling), laid out for CDNA4:
//
//   GEMM view  m = output pixel (n, oh, ow), n = output channel, k = (tap,
//              ci) with tap = 3 kh + kw: h[m][co] = sum_k A[m][k] W[k][co],
//              A[m][(tap, ci)] = x[n][ci][oh + kh - 1][ow + kw - 1] (zero
//              outside the image).  No im2col buffer exists.
//   tile       two output rows x 128 columns (256 pixels) x 128 output
//              channels per workgroup of 4 waves (2 x 2); each wave owns 64
//              columns of both rows x 64 channels = 4 x 2 blocks of
//              v_mfma_f32_32x32x16_bf16.  Row block bi holds output row
//              bi >> 1 and columns (bi & 1) * 32 .. + 31 of the wave's half,
//              so both rows and both columns of every 2x2 pooling window sit
//              in one lane's accumulators.
//   input      the tile's halo -- 4 input rows x 130 columns x 64 channels --
//              is staged once in LDS as [pixel][channel] (transposed from
//              NCHW in registers with v_perm_b32), 16-byte channel chunks
//              XOR-swizzled by pixel; every tap reads its A fragments from it
//              with a shifted pixel index.
//   weights    repacked per call by kf_conv_pack_weights to [tap][co][ci],
//              then streamed per K-step (one tap, 32 channels = 8 KiB) into
//              four LDS stages by LDS DMA, three steps ahead.
//   order      A fragment = MFMA "A" operand: each lane's accumulators are
//              runs of 4 consecutive output pixels of one channel.
#include <type_traits>

#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int NT = 256;
constexpr int CIN = 64;              // channels the halo holds
constexpr int WID = 128;             // image width (= tile width)
constexpr int COUT = 128;            // output channels (= tile width in N)
constexpr int HALO_COLS = WID + 2;   // iw = -1 .. WID
constexpr int HALO_ROWS = 4;         // ih = oh0 - 1 .. oh0 + 2
constexpr int PIX_BYTES = CIN * 2;   // 128 bytes of channels per pixel
constexpr int kHalo = HALO_ROWS * HALO_COLS * PIX_BYTES;  // 66560 bytes
constexpr int kWStage = COUT * 64;   // [128 co][32 ci] bf16 = 8 KiB
constexpr int kSteps = 9 * (CIN / 32);  // 18 K-steps of 32

#define LDS3 __attribute__((address_space(3)))

template <int V>
using IC = std::integral_constant<int, V>;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

template <typename T>
__device__ __forceinline__ T lds_load(const unsigned char* p) {
  return *reinterpret_cast<const T*>(p);
}

// byte offset of channel chunk c (8 channels) of halo pixel p
__device__ __forceinline__ uint32_t halo_off(int p, int c) { return (uint32_t)(p * PIX_BYTES + ((c ^ (p & 7)) << 4)); }

// acc[bi][bj][i]: pixel row  (bi >> 1), column wm*64 + (bi & 1)*32 + (i/4)*8 + (lane >> 5)*4 + i%4
//                 channel    wn*64 + bj*32 + (lane & 31)
typedef f32x16 CAcc[4][2];

// Element-wise ops oi..oe-1 (BIAS and the activations) on one lane's values
// of output channel `co`: the op kind is uniform, so the switch is taken once
// per op and the loop over the registers is unrolled inside each case.
template <int N>
__device__ __forceinline__ void conv_apply_phase(const ConvArgs& p, int oi, int oe, int co, float (&v)[N]) {
  for (int o = oi; o < oe; ++o) {
    const EpiOp op = p.prog.op[o];
    if (op.kind == KF_OP_BIAS) {
      const float b = p.bias[co];
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] += b;
    } else {
      apply_elementwise_array(op.kind, op.p0, op.p1, v);
    }
  }
}

}  // namespace

// wp[tap][co][ci] = w[co][ci][kh][kw]
__global__ __launch_bounds__(256) void kf_conv_pack_weights(const uint16_t* __restrict__ w, uint16_t* __restrict__ wp,
                                                            int cout, int cin) {
  const int64_t total = (int64_t)cout * cin * 9;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int ci = (int)(e % cin);
    const int co = (int)((e / cin) % cout);
    const int tap = (int)(e / ((int64_t)cin * cout));
    wp[e] = w[((int64_t)co * cin + ci) * 9 + tap];
  }
}

__global__ __launch_bounds__(NT, 1) void kf_conv3x3_bf16_256x128(ConvArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(1024))) unsigned char sHalo[kHalo];
  __shared__ __attribute__((aligned(1024))) unsigned char sW0[kWStage], sW1[kWStage], sW2[kWStage], sW3[kWStage];
  auto stW = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sW0 : S == 1 ? sW1 : S == 2 ? sW2 : sW3;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int H = (int)p.H;
  const int rows_per_img = H / 2;
  const int n_img = blockIdx.x / rows_per_img;
  const int ph = blockIdx.x % rows_per_img;  // tile = output rows 2 ph, 2 ph + 1
  const int oh0 = 2 * ph;

  // ---- stage the halo: x[n][ci][oh0-1+hr][iw] -> sHalo[(hr*130 + iw+1)][ci]
  {
    const uint16_t* X = reinterpret_cast<const uint16_t*>(p.x) + (int64_t)n_img * CIN * H * WID;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(X, (uint32_t)((int64_t)CIN * H * WID * 2));
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int b = tid + half * 256;  // block: 8 channels x 8 pixels of one row
      const int cg = b & 7, pg = (b >> 3) & 15, hr = b >> 7;
      const int ih = oh0 - 1 + hr;
      const bool row_ok = ih >= 0 && ih < H;
      u32x4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t off = row_ok ? (uint32_t)((((int64_t)(cg * 8 + j) * H + ih) * WID + pg * 8) * 2) : kOOB;
        v[j] = buf_load16(rx, off);
      }
      // 8x8 transpose of bf16: v[j] = channel cg*8+j, pixels pg*8 .. +7
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t sel = (k & 1) ? 0x07060302u : 0x05040100u;
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = __builtin_amdgcn_perm(v[2 * e + 1][k >> 1], v[2 * e][k >> 1], sel);
        const int pix = hr * HALO_COLS + pg * 8 + k + 1;
        *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = o;
      }
    }
    // zero padding columns iw = -1 and iw = WID of every halo row
    if (tid < 64) {
      const int hr = tid >> 4, side = (tid >> 3) & 1, cg = tid & 7;
      const int pix = hr * HALO_COLS + (side ? HALO_COLS - 1 : 0);
      *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = u32x4{0u, 0u, 0u, 0u};
    }
  }

  // ---- weight stream: step s = (tap s/2, channel half s%2) -> [co][32 ci]
  // stage with chunk c of row co stored at c ^ ((co >> 1) & 3); wave w fills
  // rows [32w, 32w + 32) with 2 DMA instructions of 16 rows
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)(9 * COUT * CIN * 2));
  const int dma_lc = (lane & 3) ^ ((lane >> 3) & 3);
  uint32_t vw[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int co = wave * 32 + i * 16 + (lane >> 2);
    vw[i] = (uint32_t)((co * CIN + dma_lc * 8) * 2);
  }
  auto dma_one = [&](auto S_c, auto J_c, int s) {
    constexpr int J = decltype(J_c)::value;
    const bool live = s < kSteps;
    const int soff = live ? ((s >> 1) * COUT * CIN + (s & 1) * 32) * 2 : 0;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS3 void*)(stW(S_c) + wave * 2048 + J * 1024), 16,
                                              live ? vw[J] : kOOB, soff, 0, 0);
  };

  // ---- fragment reads
  const int r32 = lane & 31, kg = lane >> 5;
  uint32_t rB[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int ch = kk * 2 + kg;
    rB[kk] = (uint32_t)((wn * 64 + r32) * 64 + ((ch ^ ((r32 >> 1) & 3)) << 4));
  }
  u32x4 fa[2][2][4], fb[2][2][2];  // [buffer][16-k half][block]
  constexpr int kReads = 12;       // per step: 8 A (4 blocks x 2 halves), 4 B
  auto read_one = [&](auto S_c, auto BUF_c, auto J_c, int s) {
    constexpr int BUF = decltype(BUF_c)::value;
    constexpr int J = decltype(J_c)::value;
    constexpr int kk = J / 6, j = J % 6;
    if constexpr (j < 4) {
      // past the last step (the prefetch of step kSteps) read the last tap
      // again: the values are never used, and the halo index stays in range
      const int sc = s < kSteps ? s : kSteps - 1;
      const int tap = sc >> 1, kh = tap / 3, kw = tap - kh * 3;
      const int pix = ((j >> 1) + kh) * HALO_COLS + wm * 64 + (j & 1) * 32 + r32 + kw;
      const int ch = (sc & 1) * 4 + kk * 2 + kg;
      fa[BUF][kk][j] = lds_load<u32x4>(sHalo + halo_off(pix, ch));
    } else {
      fb[BUF][kk][j - 4] = lds_load<u32x4>(stW(S_c) + rB[kk] + (j - 4) * 2048);
    }
  };

  CAcc acc;
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;

  constexpr int kDma = 2;
  // K-step s on weight stage S (same pipeline as the GEMM kernel): publish
  // stage S+1, then 16 MFMAs with the fragment reads of step s+1 and the
  // weight DMA of step s+3 interleaved in a fixed order.
  auto step = [&](auto S_c, auto BUF_c, int s) {
    constexpr int S = decltype(S_c)::value;
    constexpr int BUF = decltype(BUF_c)::value;
    wait_vmcnt<kDma>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, 16>([&](auto I_c) {
      constexpr int i = decltype(I_c)::value;
      constexpr int kk = i / 8, bi = (i / 2) % 4, bj = i % 2;
      acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[BUF][kk][bi]),
                                                            __builtin_bit_cast(bf16x8, fb[BUF][kk][bj]), acc[bi][bj], 0,
                                                            0, 0);
      if constexpr (i < kReads) read_one(IC<(S + 1) & 3>{}, IC<BUF ^ 1>{}, I_c, s + 1);
      if constexpr (i == 3 || i == 11) dma_one(IC<(S + 3) & 3>{}, IC<(i == 3 ? 0 : 1)>{}, s + 3);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  dma_one(IC<0>{}, IC<0>{}, 0);
  dma_one(IC<0>{}, IC<1>{}, 0);
  dma_one(IC<1>{}, IC<0>{}, 1);
  dma_one(IC<1>{}, IC<1>{}, 1);
  dma_one(IC<2>{}, IC<0>{}, 2);
  dma_one(IC<2>{}, IC<1>{}, 2);
  __syncthreads();  // halo written, first three weight stages landed
  static_for<0, kReads>([&](auto J_c) { read_one(IC<0>{}, IC<0>{}, J_c, 0); });

  // 18 steps = 4 x 4 + 2
#pragma unroll 1
  for (int s = 0; s < 16; s += 4) {
    step(IC<0>{}, IC<0>{}, s);
    step(IC<1>{}, IC<1>{}, s + 1);
    step(IC<2>{}, IC<0>{}, s + 2);
    step(IC<3>{}, IC<1>{}, s + 3);
  }
  step(IC<0>{}, IC<0>{}, 16);
  step(IC<1>{}, IC<1>{}, 17);
  __syncthreads();

  // ---- epilogue: ops before the pool on every pre-pool value, the pool in
  // registers, ops after it on the pooled values, one store
  const int nops = p.prog.n;
  const int pidx = p.pool ? p.pool_index : nops;
  const int64_t plane_out = p.pool ? (int64_t)(H / 2) * (WID / 2) : (int64_t)H * WID;
  uint16_t* out = reinterpret_cast<uint16_t*>(p.out);
  static_for<0, 2>([&](auto bj_c) {
    constexpr int bj = decltype(bj_c)::value;
    const int co = wn * 64 + bj * 32 + (lane & 31);
    uint16_t* oc = out + ((int64_t)n_img * COUT + co) * plane_out;
    float v[64];  // v[bi * 16 + i] = acc[bi][bj][i]
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int i = 0; i < 16; ++i) v[bi * 16 + i] = acc[bi][bj][i];
    conv_apply_phase(p, 0, pidx, co, v);
    if (p.pool) {
      // window (bc, q, h2): columns i, i+1 (i = 4q + 2 h2) of row blocks bc
      // (output row 0) and bc + 2 (output row 1)
      float pv[16];
#pragma unroll
      for (int bc = 0; bc < 2; ++bc)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const int i = q * 4 + h2 * 2;
            pv[bc * 8 + q * 2 + h2] = fmaxf(fmaxf(v[bc * 16 + i], v[bc * 16 + i + 1]),
                                            fmaxf(v[(bc + 2) * 16 + i], v[(bc + 2) * 16 + i + 1]));
          }
      conv_apply_phase(p, pidx + 1, nops, co, pv);
#pragma unroll
      for (int bc = 0; bc < 2; ++bc)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int pw = wm * 32 + bc * 16 + q * 4 + (lane >> 5) * 2;
          *reinterpret_cast<uint32_t*>(oc + (int64_t)ph * (WID / 2) + pw) =
              pack_bf16x2(pv[bc * 8 + q * 2], pv[bc * 8 + q * 2 + 1]);
        }
    } else {
#pragma unroll
      for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int oh = oh0 + (bi >> 1);
          const int ow = wm * 64 + (bi & 1) * 32 + q * 8 + (lane >> 5) * 4;
          const float* x = &v[bi * 16 + q * 4];
          *reinterpret_cast<u32x2*>(oc + (int64_t)oh * WID + ow) = u32x2{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
        }
    }
  });
}

hipError_t launch_conv_pack(const ConvArgs& args, void* packed_weights, hipStream_t stream) {
  hipLaunchKernelGGL(kf_conv_pack_weights, dim3(288), dim3(256), 0, stream,
                     reinterpret_cast<const uint16_t*>(args.w), reinterpret_cast<uint16_t*>(packed_weights),
                     (int)args.cout, (int)args.cin);
  return hipGetLastError();
}

hipError_t launch_conv_bf16(const ConvArgs& args, const void* packed_weights, hipStream_t stream) {
  const dim3 grid((unsigned)(args.batch * (args.H / 2)));
  hipLaunchKernelGGL(kf_conv3x3_bf16_256x128, grid, dim3(NT), 0, stream, args,
                     reinterpret_cast<const uint16_t*>(packed_weights));
  return hipGetLastError();
}

int conv_bf16_cin() { return CIN; }
int conv_bf16_width() { return WID; }
int conv_bf16_cout() { return COUT; }

}  // namespace kf
