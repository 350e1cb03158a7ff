// 3x3x3 convolution (stride 1, no padding, bf16, channels-last input, OIDHW
// weight) as an implicit GEMM on the matrix cores, with the bias, element-wise
// ops, a softmax over the output channels and two MaxPool3d(2) fused into the
// epilogue: the Conv3d -> softmax -> max-pool -> max-pool operator of the
// paper's case study (Appendix C), whose conv and pools stayed library calls
// there, as one kernel.
//
//   GEMM view  rows = the 64 output channels (2 blocks of 32), columns =
//              output positions, k = (tap, ci) with tap = 9 kd + 3 kh + kw:
//              h[co][p] = sum_k W[co][(tap, ci)] X[(tap, ci)][p] with
//              X[(tap, ci)][(od, oh, ow)] = x[od + kd][oh + kh][ow + kw][ci].
//              The weights are the MFMA A operand and the positions the B
//              operand, so a lane's accumulators are 32 channels of ONE
//              position (lane ^ 32 holds the other 32): the channel softmax is
//              in-lane arithmetic plus one exchange per reduction.
//   tile       4 x 4 x 16 output positions (d, h, w) x 64 channels per
//              workgroup of 4 waves.  Wave w owns the 4 x 4 x 4 block at
//              w = 4 w -- one cell of the two stacked 2x pools -- as two
//              column blocks of 32 positions (d pairs {0,1} and {2,3}); in a
//              block, lane bits 0-1 are w, 2-3 h, 4 the low bit of d.  Cin = 16
//              makes each tap one 16-deep MFMA step.
//   input      the tile's halo, 6 x 6 x 18 positions x 16 channels (32 bytes
//              per position), arrives in LDS by DMA as [d][h][w][2 chunks of 8
//              channels] with the chunk index XOR the parity of h, so that the
//              16 lanes of every fragment read (4 w x 4 h at one d) land on 16
//              distinct 16-byte bank slots.  Every tap reads its B fragments
//              from the same halo at a shifted position; the shift is the
//              immediate offset of the LDS read.  The next tile's halo is
//              requested as soon as the K loop has finished with the buffer,
//              and lands while the epilogue runs.
//   weights    27 x 64 x 16 bf16 (54 KiB), repacked per call by
//              kf_conv3d_pack_weights and resident in LDS for the whole
//              persistent kernel (rows XOR-swizzled like the halo).
//   schedule   persistent, two workgroups per compute unit (76 KiB of LDS
//              each): their phases drift apart, so one workgroup's epilogue
//              -- softmax and pooling, VALU work comparable to the MFMA work
//              of a tile -- runs beside the other's K loop.  In every round of
//              grid-size tiles the workgroups of one XCD take consecutive
//              tiles, which share halo rows in that XCD's L2.
#include <type_traits>

#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int NWAVE = 4;
constexpr int NT3 = 64 * NWAVE;        // 4 waves, two workgroups per CU
constexpr int CI3 = 16;                // input channels: one MFMA k-step per tap
constexpr int CO3 = 64;                // output channels: two MFMA row blocks
constexpr int TD = 4, TH = 4, TW = 16; // output tile (d, h, w)
constexpr int HDn = TD + 2, HHn = TH + 2, HWn = TW + 2;  // halo 6 x 6 x 18
constexpr int kPos = CI3 * 2;          // 32 bytes per position
constexpr int kHaloChunks = HDn * HHn * HWn * 2;        // 1296 chunks of 16 B
constexpr int kHaloDma = (kHaloChunks + 63) / 64;       // 21 DMA instructions of 1 KiB
constexpr int kHaloPerWave = (kHaloDma + NWAVE - 1) / NWAVE;  // at most 6 (wave 0: 6, the others 5)
constexpr int kHaloBytes = kHaloDma * 1024;             // 21504
constexpr int kWBytes = 27 * CO3 * kPos;                // 55296
constexpr int kWDma = kWBytes / 1024;                   // 54
constexpr int kWPerWave = (kWDma + NWAVE - 1) / NWAVE;  // 14
constexpr int kTapStride = CO3 * kPos;                  // 2048 bytes of weights per tap
constexpr int kPbOff = 2 * HHn * HWn * kPos;            // 6912: column block 1 is d + 2
static_assert(kHaloBytes >= TD * TH * TW * 32 * 2, "the halo buffer holds one 32-channel staging pass");
static_assert(2 * (kWBytes + kHaloBytes + 1024) <= 160 * 1024, "two workgroups fit one CU's LDS");
static_assert(((2 * HHn + 2) * HWn + 2) * kPos + kPbOff < 65536, "tap offsets fit the LDS read's immediate");

#define LDS3 __attribute__((address_space(3)))

template <int V>
using IC = std::integral_constant<int, V>;

template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0x0 << 8) | ((N >> 4) << 14));
}

template <typename T>
__device__ __forceinline__ T lds_load(const unsigned char* p) {
  return *reinterpret_cast<const T*>(p);
}

// output channel held in accumulator register v of row block cb by a lane
// of half kg (lane >> 5)
__device__ __forceinline__ int acc_channel(int cb, int v, int kg) { return cb * 32 + (v >> 2) * 8 + kg * 4 + (v & 3); }

// DPP lane exchanges inside rows of 16 lanes (each pairs a lane with one
// whose bit b differs): xor 1, xor 2 (quad permutations), and the
// half-row / row mirrors, which pair lane i with 7 - i / 15 - i
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// lane ^ 16 inside each 32-lane half (ds_swizzle, bit-mask mode)
__device__ __forceinline__ float swz_xor16(float v) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (16 << 10)));
}

}  // namespace

// wp[tap][co][chunk ^ ((co >> 3) & 1)][8] = w[co][8 chunk + e][tap]: one
// thread per (co, ci) reads its 27 contiguous taps.
__global__ __launch_bounds__(256) void kf_conv3d_pack_weights(const uint16_t* __restrict__ w,
                                                              uint16_t* __restrict__ wp) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= CO3 * CI3) return;
  const int co = e / CI3, ci = e % CI3;
  const int chunk = (ci >> 3) ^ ((co >> 3) & 1);
#pragma unroll
  for (int tap = 0; tap < 27; ++tap) wp[((tap * CO3 + co) * 2 + chunk) * 8 + (ci & 7)] = w[e * 27 + tap];
}

template <int CH>
__global__ __launch_bounds__(NT3, 2) void kf_conv3d_bf16_64x256(Conv3dArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(1024))) unsigned char sW[kWBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char sH[kHaloBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char sDummy[1024];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31, kg = lane >> 5;
  const int D = p.D, H = p.H, W = p.W;
  const int64_t img_elems = (int64_t)D * H * W * CI3;
  const uint32_t img_bytes = (uint32_t)(img_elems * 2);  // < 2^30, checked by the host

  // round r of the persistent loop: the workgroups of XCD (b % 8) take
  // consecutive tiles
  const int G = p.grid;
  const int slot =
      (p.xcd_remap && (G & 7) == 0) ? (int)(blockIdx.x & 7) * (G >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
  auto tile_at = [&](int round) { return round * G + slot; };
  int t = tile_at(0);
  if (t >= p.tiles) return;

  struct TileXY {
    int n, td, th, tw;
  };
  auto coords = [&](int tt) {
    TileXY c;
    c.tw = tt % p.tiles_w;
    tt /= p.tiles_w;
    c.th = tt % p.tiles_h;
    tt /= p.tiles_h;
    c.td = tt % p.tiles_d;
    c.n = tt / p.tiles_d;
    return c;
  };

  // ---- halo DMA: instruction j (= wave + 4 i) fills LDS chunks [64 j, 64 j
  // + 64) of a halo buffer; chunk q holds position q >> 1 = (hd, hh, hw),
  // channels 8 ((q & 1) ^ (hh & 1)) .. + 7.  The per-lane offsets relative to
  // the tile origin are the same for every tile; the origin itself is the
  // scalar offset.  Positions past the volume read zeros (buffer range
  // check) or the next row's values, which only reach outputs that are never
  // stored.
  uint32_t hoff[kHaloPerWave];
#pragma unroll
  for (int i = 0; i < kHaloPerWave; ++i) {
    const int q = (wave + NWAVE * i) * 64 + lane;
    if (q < kHaloChunks) {
      const int pos = q >> 1, hw = pos % HWn, hh = (pos / HWn) % HHn, hd = pos / (HWn * HHn);
      const int cg = (q & 1) ^ (hh & 1);
      hoff[i] = (uint32_t)((((hd * H + hh) * W + hw) * CI3 + cg * 8) * 2);
    } else {
      hoff[i] = kOOB;
    }
  }
  const uint16_t* x = reinterpret_cast<const uint16_t*>(p.x);
  auto halo_dma = [&](unsigned char* buf, int tt) {
    const TileXY c = coords(tt);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + (int64_t)c.n * img_elems, img_bytes);
    const uint32_t soff = (uint32_t)(((((int64_t)c.td * TD * H + c.th * TH) * W + c.tw * TW) * CI3) * 2);
    // the waits before the K loop leave nothing of the halo in flight, so
    // the waves issue only their real instructions (an out-of-range DMA
    // instruction would still cost its issue and a 1 KiB LDS write)
#pragma unroll
    for (int i = 0; i < kHaloPerWave; ++i) {
      const int j = wave + NWAVE * i;
      if (j < kHaloDma)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS3 void*)(buf + j * 1024), 16, hoff[i], soff, 0, 0);
    }
  };

  // ---- bias of this lane's 32 channels, then the weights and the first halo
  float bv[2][16];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int v = 0; v < 16; ++v) bv[cb][v] = p.bias ? p.bias[acc_channel(cb, v, kg)] : 0.0f;
  // a bias directly followed by the softmax enters it as (h + b) log2 e =
  // fma(h, log2 e, b log2 e)
  float bl[2][16];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int v = 0; v < 16; ++v) bl[cb][v] = bv[cb][v] * kLog2e;
  {
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)kWBytes);
#pragma unroll
    for (int i = 0; i < kWPerWave; ++i) {
      const int j = wave + NWAVE * i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS3 void*)(j < kWDma ? sW + j * 1024 : sDummy), 16,
                                                j < kWDma ? (uint32_t)(j * 1024 + lane * 16) : kOOB, 0, 0, 0);
    }
  }
  halo_dma(sH, t);

  const OpTable ops = load_op_table(p.prog, lane);

  // ---- fragment addresses
  // A (weights): row co = cb * 32 + r32, chunk kg at kg ^ ((co >> 3) & 1);
  // + tap * 2048 + cb * 1024
  const uint32_t a_base = (uint32_t)(r32 * kPos + ((kg ^ ((r32 >> 3) & 1)) << 4));
  // B (positions): (d, h, w) = (r32 >> 4, (r32 >> 2) & 3, 4 wave + (r32 & 3));
  // chunk kg at kg ^ ((h + kh) & 1); + tap shift, + kPbOff for column block 1
  const int ld = r32 >> 4, lh = (r32 >> 2) & 3, lw = 4 * wave + (r32 & 3);
  const uint32_t b_pos = (uint32_t)(((ld * HHn + lh) * HWn + lw) * kPos);
  const uint32_t b_even = b_pos + ((kg ^ (lh & 1)) << 4);
  const uint32_t b_odd = b_pos + ((kg ^ (lh & 1) ^ 1) << 4);

  for (int it = 0;; ++it) {
    const int t_next = tile_at(it + 1);
    const bool has_next = t_next < p.tiles;
    // this tile's halo has landed (every wave waited for its own DMA, the
    // barrier publishes all of them); the epilogue's one output store of the
    // previous tile may still be in flight
    if (p.pools == 2 && it > 0)
      wait_vmcnt_lgkm0<1>();
    else
      wait_vmcnt_lgkm0<0>();
    __syncthreads();

    // ---- K loop: 27 taps x (2 A + 2 B fragment reads, 4 MFMAs)
    f32x16 acc[2][2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[cb][pb][v] = 0.0f;
    const unsigned char* hb_even = sH + b_even;
    const unsigned char* hb_odd = sH + b_odd;
    const unsigned char* wb = sW + a_base;
    // fragments of tap t + 1 are read while the MFMAs of tap t run (two
    // register buffers; the scheduling barriers keep that order)
    u32x4 fa[2][2], fb[2][2];
    auto read_tap = [&](auto T_c) {
      constexpr int tap = decltype(T_c)::value, buf = tap & 1;
      constexpr int kd = tap / 9, kh = (tap / 3) % 3, kw = tap % 3;
      constexpr int toff = ((kd * HHn + kh) * HWn + kw) * kPos;
      const unsigned char* hb = (kh & 1) ? hb_odd : hb_even;
      fa[buf][0] = lds_load<u32x4>(wb + tap * kTapStride);
      fa[buf][1] = lds_load<u32x4>(wb + tap * kTapStride + 32 * kPos);
      fb[buf][0] = lds_load<u32x4>(hb + toff);
      fb[buf][1] = lds_load<u32x4>(hb + toff + kPbOff);
    };
    read_tap(IC<0>{});
    __builtin_amdgcn_s_setprio(2);  // the K loop's MFMA issue goes first; the other workgroup's epilogue fills in
    static_for<0, 27>([&](auto T_c) {
      constexpr int tap = decltype(T_c)::value, buf = tap & 1;
      if constexpr (tap + 1 < 27) read_tap(IC<tap + 1>{});
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
          acc[cb][pb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[buf][cb]),
                                                                __builtin_bit_cast(bf16x8, fb[buf][pb]), acc[cb][pb],
                                                                0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    });

    __builtin_amdgcn_s_setprio(0);
    // ---- epilogue: x[cb][pb][v] = channel acc_channel(cb, v, kg) at
    // position (pb, r32).  With pooling, the halo buffer is free once every
    // wave has left the K loop, and the next tile's halo is requested now;
    // without, the buffer first serves as the staging area of the stores.
    if (p.pools == 2) {
      __syncthreads();
      if (has_next) halo_dma(sH, t_next);
    }
    float xv[2][2][16];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int v = 0; v < 16; ++v) xv[cb][pb][v] = acc[cb][pb][v];

    auto add_bias = [&]() {
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int v = 0; v < 16; ++v) xv[cb][pb][v] += bv[cb][v];
    };
    // softmax over the 64 channels of each of the lane's two positions, in
    // base 2: y = h log2 e (with_bias: (h + b) log2 e as one fma), then
    // 2^(y - max y) / sum 2^(y - max y)
    auto channel_softmax = [&](bool with_bias) {
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            xv[cb][pb][v] = with_bias ? fmaf(xv[cb][pb][v], kLog2e, bl[cb][v]) : xv[cb][pb][v] * kLog2e;
#pragma unroll
      for (int pb = 0; pb < 2; ++pb) {
        float m = xv[0][pb][0];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int v = 0; v < 16; ++v) m = fmaxf(m, xv[cb][pb][v]);
        m = fmaxf(m, shfl_xor(m, 32));
        float s = 0.0f;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            xv[cb][pb][v] = __builtin_amdgcn_exp2f(xv[cb][pb][v] - m);
            s += xv[cb][pb][v];
          }
        s += shfl_xor(s, 32);
        const float inv = frcp(s);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
          for (int v = 0; v < 16; ++v) xv[cb][pb][v] *= inv;
      }
    };
    auto elementwise = [&](int kind, int o) {
      const float p0 = op_p0(ops, o), p1 = op_p1(ops, o);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) apply_elementwise_array(kind, p0, p1, xv[cb][pb]);
    };
    if constexpr (CH == 0) {
      for (int o = 0; o < p.prog.n; ++o) {
        const int kind = op_kind(ops, o);
        if (kind == KF_OP_MAXPOOL3D_2) break;  // the pools are the trailing ops
        if (kind == KF_OP_BIAS) {
          if (o + 1 < p.prog.n && op_kind(ops, o + 1) == KF_OP_CHANNEL_SOFTMAX) {
            channel_softmax(true);
            ++o;
          } else {
            add_bias();
          }
        } else if (kind == KF_OP_CHANNEL_SOFTMAX) {
          channel_softmax(false);
        } else {
          elementwise(kind, o);
        }
      }
    } else {
      static_for<0, kChainLen[CH]>([&](auto O_c) {
        constexpr int o = decltype(O_c)::value;
        constexpr int kind = kChainOps[CH][o];
        constexpr bool fused = kind == KF_OP_BIAS && o + 1 < kChainLen[CH] && kChainOps[CH][o + 1] == KF_OP_CHANNEL_SOFTMAX;
        constexpr bool after_bias = o > 0 && kChainOps[CH][o > 0 ? o - 1 : 0] == KF_OP_BIAS;
        if constexpr (fused)
          channel_softmax(true);
        else if constexpr (kind == KF_OP_BIAS)
          add_bias();
        else if constexpr (kind == KF_OP_CHANNEL_SOFTMAX && !after_bias)
          channel_softmax(false);
        else if constexpr (kind != KF_OP_MAXPOOL3D_2 && kind != KF_OP_CHANNEL_SOFTMAX)
          elementwise(kind, o);
      });
    }

    const TileXY c = coords(t);
    uint16_t* out = reinterpret_cast<uint16_t*>(p.out);
    if (p.pools == 2) {
      // max over the wave's 4 x 4 x 4 block: the two column blocks in-lane,
      // then a reduce-scatter over lane bits 4..0 (the positions) -- at each
      // step a lane keeps half of its values and takes the maximum with its
      // partner's copy of that half -- so that lane r32 ends with the block
      // maximum of value index r32 = (cb, v)
      // A compiled chain whose last op before the pools is the softmax pools
      // values that are finite and >= +0, whose order is that of their bit
      // patterns as unsigned integers: the integer maximum picks the same
      // value without the NaN quieting a float maximum needs.
      constexpr bool kIntMax = CH != 0 && kChainOps[CH][kChainLen[CH] > 2 ? kChainLen[CH] - 3 : 0] == KF_OP_CHANNEL_SOFTMAX;
      auto vmax = [](float a, float b) {
        if constexpr (kIntMax)
          return __uint_as_float(max(__float_as_uint(a), __float_as_uint(b)));
        else
          return fmaxf(a, b);
      };
      float y[32];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int v = 0; v < 16; ++v) y[cb * 16 + v] = vmax(xv[cb][0][v], xv[cb][1][v]);
      // lane bit 4: ds_swizzle exchanges the half a lane gives away
      {
        const bool up = (r32 & 16) != 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float send = up ? y[i] : y[i + 16];
          const float keep = up ? y[i + 16] : y[i];
          y[i] = vmax(keep, swz_xor16(send));
        }
      }
      // lane bits 3..0: the partner's value comes by DPP; both halves are
      // combined and the lane keeps its own
      auto step = [&](auto M_c, auto CTRL_c) {
        constexpr int mask = decltype(M_c)::value, ctrl = decltype(CTRL_c)::value;
        const bool up = (r32 & mask) != 0;
#pragma unroll
        for (int i = 0; i < mask; ++i) {
          const float lo = vmax(y[i], dpp<ctrl>(y[i]));
          const float hi = vmax(y[i + mask], dpp<ctrl>(y[i + mask]));
          y[i] = up ? hi : lo;
        }
      };
      step(IC<8>{}, IC<kDppMirror>{});
      step(IC<4>{}, IC<kDppHalfMirror>{});
      step(IC<2>{}, IC<kDppXor2>{});
      step(IC<1>{}, IC<kDppXor1>{});
      // one store instruction per wave whatever the window (a window past
      // the output stores nothing: its offset is out of range), so that the
      // next tile's wait can leave exactly this store in flight
      const int pd = c.td, ph = c.th, pw = c.tw * 4 + wave;
      const int64_t per_img = (int64_t)CO3 * p.Dp * p.Hp * p.Wp;
      const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + (int64_t)c.n * per_img, (uint32_t)(per_img * 2));
      const int ch = acc_channel(r32 >> 4, r32 & 15, kg);
      const bool live = pd < p.Dp && ph < p.Hp && pw < p.Wp;
      const uint32_t off = live ? (uint32_t)((((int64_t)ch * p.Dp + pd) * p.Hp + ph) * p.Wp + pw) * 2u : kOOB;
      __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f32_to_bf16_rne(y[0]), ro, off, 0, 0);
    } else {
      // every position: stage 32 channels x 256 positions of bf16 in the
      // halo buffer (free once every wave has left the K loop), then write
      // rows of 16 w per (channel, d, h)
      __syncthreads();
      unsigned char* stage = sH;
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int chl = (v >> 2) * 8 + kg * 4 + (v & 3);
            const int pos = ((2 * pb + ld) * TH + lh) * TW + lw;
            *reinterpret_cast<uint16_t*>(stage + (chl * (TD * TH * TW) + pos) * 2) =
                (uint16_t)f32_to_bf16_rne(xv[cb][pb][v]);
          }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 32 * TD * TH * 2 / NT3; ++k) {
          const int q = tid + NT3 * k;  // 16-byte chunk: row q >> 1 = (channel, d, h), half q & 1
          const int row = q >> 1, half = q & 1;
          const int chl = row >> 4, od = c.td * TD + ((row >> 2) & 3), oh = c.th * TH + (row & 3);
          const int ow = c.tw * TW + half * 8;
          if (od < p.Dp && oh < p.Hp && ow < p.Wp) {
            const u32x4 w4 = *reinterpret_cast<const u32x4*>(stage + row * 32 + half * 16);
            uint16_t* dst = out + ((((int64_t)c.n * CO3 + cb * 32 + chl) * p.Dp + od) * p.Hp + oh) * p.Wp + ow;
            if ((p.Wp & 7) == 0 && ow + 8 <= p.Wp) {
              *reinterpret_cast<u32x4*>(dst) = w4;
            } else {
#pragma unroll
              for (int e = 0; e < 8; ++e)
                if (ow + e < p.Wp) dst[e] = (uint16_t)((e & 1) ? (w4[e >> 1] >> 16) : (w4[e >> 1] & 0xffffu));
            }
          }
        }
        __syncthreads();
      }
      if (has_next) halo_dma(sH, t_next);
    }
    if (!has_next) break;
    t = t_next;
  }
  // nothing may land in LDS after the workgroup ends
  wait_vmcnt_lgkm0<0>();
}

hipError_t launch_conv3d_pack(const void* w, void* packed_weights, hipStream_t stream) {
  hipLaunchKernelGGL(kf_conv3d_pack_weights, dim3((CO3 * CI3 + 255) / 256), dim3(256), 0, stream,
                     reinterpret_cast<const uint16_t*>(w), reinterpret_cast<uint16_t*>(packed_weights));
  return hipGetLastError();
}

hipError_t launch_conv3d_bf16(const Conv3dArgs& args, const void* packed_weights, int chain, hipStream_t stream) {
  if (args.tiles <= 0) return hipSuccess;
  const dim3 grid((unsigned)(args.grid < args.tiles ? args.grid : args.tiles));
  Conv3dArgs a = args;
  a.grid = (int)grid.x;
  const uint16_t* wp = reinterpret_cast<const uint16_t*>(packed_weights);
  if (chain == 10)
    hipLaunchKernelGGL(kf_conv3d_bf16_64x256<10>, grid, dim3(NT3), 0, stream, a, wp);
  else if (chain == 1)
    hipLaunchKernelGGL(kf_conv3d_bf16_64x256<1>, grid, dim3(NT3), 0, stream, a, wp);
  else
    hipLaunchKernelGGL(kf_conv3d_bf16_64x256<0>, grid, dim3(NT3), 0, stream, a, wp);
  return hipGetLastError();
}

int conv3d_cin() { return CI3; }
int conv3d_cout() { return CO3; }
size_t conv3d_packed_bytes() { return (size_t)kWBytes; }

}  // namespace kf
