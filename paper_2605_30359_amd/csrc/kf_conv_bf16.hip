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
//              three LDS stages by LDS DMA, three steps ahead.
//   schedule   persistent: one workgroup per compute unit walks the tiles
//              with a stride of the grid size.  The next tile's halo rows
//              arrive by LDS DMA spread over the current tile's K-steps and
//              are transposed at the boundary, and the weight stream runs on
//              across tiles, so neither waits at a tile boundary.
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
constexpr int HALO_SLOTS = 4;        // input rows the halo holds (a ring)
constexpr int PIX_BYTES = CIN * 2;   // 128 bytes of channels per pixel
constexpr int kSlot = HALO_COLS * PIX_BYTES;  // one input row of the halo: 16640 bytes
constexpr int kHalo = HALO_SLOTS * kSlot;     // 66560 bytes
constexpr int kWStage = COUT * 64;   // [128 co][32 ci] bf16 = 8 KiB
constexpr int kWS = 6;               // weight stages = prefetch distance in K-steps
constexpr int kRaw = CIN * 2 * WID * 2;  // two input rows as loaded: [ci][2 rows][128 px] = 32 KiB
constexpr int kRawDma = kRaw / 1024 / 4;  // DMA instructions per wave for two input rows
constexpr int kSteps = 9 * (CIN / 32);  // 18 K-steps of 32 per tile
static_assert(kSteps % kWS == 0 && kSteps % 2 == 0, "a tile's steps cycle whole weight stages and fragment buffers");
// the next tile's rows go out on the even K-steps 0, 2, .., 2 (kRawDma - 1)
static_assert(kSteps == 18 && kWS == 6 && kRawDma == 8, "the DMA wait counts below are derived for this schedule");

#define LDS3 __attribute__((address_space(3)))

template <int V>
using IC = std::integral_constant<int, V>;

// s_waitcnt vmcnt(N) lgkmcnt(0), expcnt left alone
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0x0 << 8) | ((N >> 4) << 14));
}

template <typename T>
__device__ __forceinline__ T lds_load(const unsigned char* p) {
  return *reinterpret_cast<const T*>(p);
}

// byte offset of channel chunk c (8 channels) of halo pixel p: a 16-lane
// fragment read covers 16 consecutive pixels, whose chunks land on the 16
// distinct 16-byte slots of a 256-byte bank line (pixel parity picks the
// half, bits 1-3 of the pixel the chunk swizzle)
__device__ __forceinline__ uint32_t halo_off(int p, int c) {
  return (uint32_t)(p * PIX_BYTES + ((c ^ ((p >> 1) & 7)) << 4));
}

// acc[bi][bj][i]: pixel row  (bi >> 1), column wm*64 + (bi & 1)*32 + (i/4)*8 + (lane >> 5)*4 + i%4
//                 channel    wn*64 + bj*32 + (lane & 31)
typedef f32x16 CAcc[4][2];

// Element-wise ops oi..oe-1 (BIAS and the activations) on one lane's values
// of one output channel, whose bias is b: the op kind is uniform, so the
// switch is taken once per op and the loop over the registers is unrolled
// inside each case.
template <int N>
__device__ __forceinline__ void conv_apply_op(const OpTable& ops, int kind, int o, float b, float (&v)[N]) {
  if (kind == KF_OP_BIAS) {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] += b;
  } else {
    apply_elementwise_array(kind, op_p0(ops, o), op_p1(ops, o), v);
  }
}
template <int CH, int N>
__device__ __forceinline__ void conv_apply_phase(const OpTable& ops, int oi, int oe, float b, float (&v)[N]) {
  if constexpr (CH == 0) {
    for (int o = oi; o < oe; ++o) conv_apply_op(ops, op_kind(ops, o), o, b, v);
  } else {
    static_for<0, kChainLen[CH]>([&](auto O_c) {
      constexpr int o = decltype(O_c)::value;
      if (o >= oi && o < oe) conv_apply_op(ops, kChainOps[CH][o], o, b, v);
    });
  }
}

// A compile-time chain whose ops before the pool are all non-decreasing and
// exact in floating point (bias add, ReLU, hardtanh) can pool first: max
// commutes with each of them, so the result is the same bit for bit, and
// the ops run on a quarter of the values.
constexpr bool chain_pools_first(int ch) {
  if (ch == 0) return false;
  for (int o = 0; o < kChainLen[ch]; ++o) {
    const int k = kChainOps[ch][o];
    if (k == KF_OP_MAXPOOL2X2) return true;
    if (k != KF_OP_BIAS && k != KF_OP_RELU && k != KF_OP_HARDTANH) return false;
  }
  return false;
}

}  // namespace

// wp[tap][co][ci] = w[co][ci][kh][kw]: one thread per (co, ci) reads its 9
// contiguous taps and writes them to the 9 tap planes, so that a wave's reads
// and each of its writes cover contiguous memory.
__global__ __launch_bounds__(256) void kf_conv_pack_weights(const uint16_t* __restrict__ w, uint16_t* __restrict__ wp,
                                                            int cout, int cin) {
  const int64_t pairs = (int64_t)cout * cin;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < pairs; e += (int64_t)gridDim.x * 256) {
    uint16_t t[9];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) t[tap] = w[e * 9 + tap];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) wp[tap * pairs + e] = t[tap];
  }
}

template <int CH>
__global__ __launch_bounds__(NT, 1) void kf_conv3x3_bf16_256x128(ConvArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(1024))) unsigned char sHalo[kHalo];
  __shared__ __attribute__((aligned(1024))) unsigned char sRaw[kRaw];
  __shared__ __attribute__((aligned(1024))) unsigned char sW0[kWStage], sW1[kWStage], sW2[kWStage], sW3[kWStage],
      sW4[kWStage], sW5[kWStage];
  __shared__ __attribute__((aligned(1024))) unsigned char sDummy[1024];
  auto stW = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sW0 : S == 1 ? sW1 : S == 2 ? sW2 : S == 3 ? sW3 : S == 4 ? sW4 : sW5;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int H = (int)p.H;
  const int rows_per_img = H / 2;
  const int64_t img_elems = (int64_t)CIN * H * WID;

  // ---- halo: a ring of 4 input rows, slot k at sHalo + k * kSlot, each as
  // [130 pixels (iw = -1 .. WID)][64 channels].  Logical row lr (input row
  // oh0 - 1 + lr) of the current tile sits in slot (rb + lr) & 3.  A
  // workgroup walks a contiguous range of tiles; the next tile of the same
  // image shares two input rows with this one, so only two new rows are
  // loaded per tile (rb advances by 2), and only at the start of the range
  // or of an image are all four loaded.
  //
  // Two input rows of every channel arrive by LDS DMA into sRaw as [ci][2
  // rows][128 px] (row (ci, r) = 256 bytes, its 16-byte chunk q stored at q ^
  // rsw(ci)); at the tile boundary each thread transposes one block of 8
  // channels x 8 pixels from sRaw into its halo slot with v_perm_b32.  Wave
  // w's DMA i (0 .. 7) fetches channels 2 (8 w + i) and 2 (8 w + i) + 1, lane
  // l channel 2 (8 w + i) + (l >> 5), row (l >> 4) & 1, chunk position l & 15.
  auto rsw = [](int c) { return ((c >> 3) << 1) & 15; };
  auto raw_dma = [&](int i, int n_img, int ih0, bool live) {
    const int c = 2 * (wave * kRawDma + i) + (lane >> 5);
    const int ih = ih0 + ((lane >> 4) & 1);
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(reinterpret_cast<const uint16_t*>(p.x) + (live ? n_img : 0) * img_elems, (uint32_t)(img_elems * 2));
    const int q = (lane & 15) ^ rsw(c);
    const bool ok = live && ih >= 0 && ih < H;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS3 void*)(live ? sRaw + (wave * kRawDma + i) * 1024 : sDummy), 16,
                                              ok ? (uint32_t)(((c * H + ih) * WID + q * 8) * 2) : kOOB, 0, 0, 0);
  };
  // sRaw -> halo slots s0 (its row 0) and s1 (row 1), zero padding columns
  auto halo_write = [&](int s0, int s1) {
    {
      const int cg = tid & 7, pg = (tid >> 3) & 15, r = tid >> 7;
      const int slot = r ? s1 : s0;
      u32x4 hv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = cg * 8 + j;
        hv[j] = *reinterpret_cast<const u32x4*>(sRaw + c * 512 + r * 256 + ((pg ^ rsw(c)) << 4));
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t sel = (k & 1) ? 0x07060302u : 0x05040100u;
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = __builtin_amdgcn_perm(hv[2 * e + 1][k >> 1], hv[2 * e][k >> 1], sel);
        const int pix = slot * HALO_COLS + pg * 8 + k + 1;
        *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = o;
      }
    }
    if (tid < 32) {
      const int r = tid >> 4, side = (tid >> 3) & 1, cg = tid & 7;
      const int pix = (r ? s1 : s0) * HALO_COLS + (side ? HALO_COLS - 1 : 0);
      *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = u32x4{0u, 0u, 0u, 0u};
    }
  };

  // ---- weight stream: step s = (tap s/2, channel half s%2) -> [co][32 ci]
  // stage with chunk c of row co stored at c ^ ((co >> 2) & 3) (16
  // consecutive rows of a fragment read on 16 distinct bank slots); wave w fills
  // rows [32w, 32w + 32) with 2 DMA instructions of 16 rows.  The weights
  // are the same for every tile, so the stream runs on across tiles: the
  // DMA issued in step s of a tile fetches step (s + 6) mod 18, for this tile
  // or the next.
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)(9 * COUT * CIN * 2));
  const int dma_lc = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t vw[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int co = wave * 32 + i * 16 + (lane >> 2);
    vw[i] = (uint32_t)((co * CIN + dma_lc * 8) * 2);
  }
  auto dma_one = [&](auto S_c, auto J_c, int s, bool live) {
    constexpr int J = decltype(J_c)::value;
    const int sw = s >= kSteps ? s - kSteps : s;
    const int soff = ((sw >> 1) * COUT * CIN + (sw & 1) * 32) * 2;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS3 void*)(stW(S_c) + wave * 2048 + J * 1024), 16,
                                              live ? vw[J] : kOOB, soff, 0, 0);
  };

  // ---- fragment reads
  const int r32 = lane & 31, kg = lane >> 5;
  uint32_t rB[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int ch = kk * 2 + kg;
    rB[kk] = (uint32_t)((wn * 64 + r32) * 64 + ((ch ^ ((r32 >> 2) & 3)) << 4));
  }
  int rb = 0;                      // ring slot of logical halo row 0
  u32x4 fa[2][2][4], fb[2][2][2];  // [buffer][16-k half][block]
  constexpr int kReads = 12;       // per step: 8 A (4 blocks x 2 halves), 4 B
  auto read_one = [&](auto S_c, auto BUF_c, auto J_c, int s) {
    constexpr int BUF = decltype(BUF_c)::value;
    constexpr int J = decltype(J_c)::value;
    constexpr int kk = J / 6, j = J % 6;
    if constexpr (j < 4) {
      // past the last step (the read ahead of step kSteps) read the last tap
      // again: the values are never used, and the halo index stays in range
      const int sc = s < kSteps ? s : kSteps - 1;
      const int tap = sc >> 1, kh = tap / 3, kw = tap - kh * 3;
      const int slot = (rb + (j >> 1) + kh) & 3;
      const int pix = slot * HALO_COLS + wm * 64 + (j & 1) * 32 + r32 + kw;
      const int ch = (sc & 1) * 4 + kk * 2 + kg;
      fa[BUF][kk][j] = lds_load<u32x4>(sHalo + halo_off(pix, ch));
    } else {
      fb[BUF][kk][j - 4] = lds_load<u32x4>(stW(S_c) + rB[kk] + (j - 4) * 2048);
    }
  };

  // bias of this lane's two output channels, once for all tiles
  float bias_v[2] = {0.0f, 0.0f};
  if (p.bias) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) bias_v[bj] = p.bias[wn * 64 + bj * 32 + (lane & 31)];
  }

  CAcc acc;
  // K-step s of a tile on weight stage S = s % 6: every wave has read its
  // fragments of stage S (during step s-1) once it passes the barrier, so the
  // DMA of step s+6 goes into stage S; the barrier also publishes stage S+1
  // (DMA issued during step s-5), read during this step.  Each step issues
  // its 2 weight DMA instructions, and the even steps one row DMA after them
  // (rows 0..7 on steps 0..14, a dummy on step 16): an LDS DMA instruction
  // costs its issue slot and an LDS write even out of range, so there is no
  // dummy on the odd steps.  A wave's loads complete in issue order, so the
  // wait for stage S+1 leaves in flight exactly what was issued after it: the
  // row DMA of step s-5 if s-5 is even, and the 8 weight and 2 row DMAs of
  // steps s-4 .. s-1 -- 10 or 11 instructions, by the parity of s (= that of
  // S); it also covers the rows requested up to step s-6, whose HBM latency
  // is thereby hidden behind five K-steps.
  // the next tile's rows: image n_next, first input row ih_next (rows_live: any)
  auto step = [&](auto S_c, auto BUF_c, int s, bool next_live, bool rows_live, int n_next, int ih_next) {
    constexpr int S = decltype(S_c)::value;
    constexpr int BUF = decltype(BUF_c)::value;
    wait_vmcnt_lgkm0<(S & 1) ? 11 : 10>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const bool live = s + kWS < kSteps || next_live;
    static_for<0, 16>([&](auto I_c) {
      constexpr int i = decltype(I_c)::value;
      constexpr int kk = i / 8, bi = (i / 2) % 4, bj = i % 2;
      acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[BUF][kk][bi]),
                                                            __builtin_bit_cast(bf16x8, fb[BUF][kk][bj]), acc[bi][bj], 0,
                                                            0, 0);
      if constexpr (i < kReads) read_one(IC<(S + 1) % kWS>{}, IC<BUF ^ 1>{}, I_c, s + 1);
      if constexpr (i == 1 || i == 3) dma_one(S_c, IC<(i == 1 ? 0 : 1)>{}, s + kWS, live);
      if constexpr (i == 5 && S % 2 == 0) raw_dma(s / 2 < kRawDma ? s / 2 : 0, n_next, ih_next, rows_live && s / 2 < kRawDma);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const int pidx = p.pool ? p.pool_index : nops;
  const int64_t plane_out = p.pool ? (int64_t)(H / 2) * (WID / 2) : (int64_t)H * WID;
  uint16_t* out = reinterpret_cast<uint16_t*>(p.out);

  // this workgroup's tiles (the grid never exceeds the tile count)
  const int t_begin = (int)((int64_t)blockIdx.x * p.tiles / gridDim.x);
  const int t_end = (int)((int64_t)(blockIdx.x + 1) * p.tiles / gridDim.x);
  // tile t continues tile t-1 (same image, next row pair) inside the range
  auto continues = [&](int t) { return t > t_begin && t % rows_per_img != 0; };

  // prologue: input rows 0-1 of the first tile, then the weight stages of
  // steps 0-5, issued as K-steps -6 .. -1 would issue them (a dummy row DMA
  // after the even ones), so that the wait counts hold from step 0 on
  for (int i = 0; i < kRawDma; ++i) raw_dma(i, t_begin / rows_per_img, 2 * (t_begin % rows_per_img) - 1, true);
  static_for<0, kWS>([&](auto S_c) {
    dma_one(S_c, IC<0>{}, decltype(S_c)::value, true);
    dma_one(S_c, IC<1>{}, decltype(S_c)::value, true);
    if constexpr (decltype(S_c)::value % 2 == 0) raw_dma(0, 0, 0, false);
  });

  for (int tile = t_begin; tile < t_end; ++tile) {
    const int n_img = tile / rows_per_img;
    const int ph = tile % rows_per_img;  // tile = output rows 2 ph, 2 ph + 1
    const int oh0 = 2 * ph;
    const bool cont = continues(tile);
    const int next_tile = tile + 1;
    const bool next_live = next_tile < t_end;
    // rows the next tile needs from sRaw: its rows 2-3 if it continues this
    // one, else its rows 0-1 (rows 2-3 follow at its boundary)
    const bool next_cont = next_live && continues(next_tile);
    const int n_next = next_tile / rows_per_img;
    const int ih_next = 2 * (next_tile % rows_per_img) + (next_cont ? 1 : -1);

    // This tile's new input rows and weight stages 0-2 have landed: only the
    // 7 DMA instructions issued after the last row request (step 14) -- the
    // weights of steps 15-17 and the dummy of step 16 -- and the previous
    // tile's output stores may still be in flight.  Every wave is past its
    // last read of the slots rewritten here and of the previous tile's output
    // staging.
    wait_vmcnt_lgkm0<7>();
    __syncthreads();
    rb = cont ? (rb + 2) & 3 : 0;
    if (cont) {
      halo_write((rb + 2) & 3, (rb + 3) & 3);
    } else {
      // start of the range or of an image: rows 0-1 are in sRaw; rows 2-3
      // are requested now and waited for
      halo_write(0, 1);
      __syncthreads();
      for (int i = 0; i < kRawDma; ++i) raw_dma(i, n_img, oh0 + 1, true);
      wait_vmcnt_lgkm0<0>();
      __syncthreads();
      halo_write(2, 3);
    }
    __syncthreads();
    static_for<0, kReads>([&](auto J_c) { read_one(IC<0>{}, IC<0>{}, J_c, 0); });

#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;

    // 18 steps = 3 x 6 (stage s % 6, fragment buffer s % 2)
#pragma unroll 1
    for (int s = 0; s < kSteps; s += 6) {
      step(IC<0>{}, IC<0>{}, s, next_live, next_live, n_next, ih_next);
      step(IC<1>{}, IC<1>{}, s + 1, next_live, next_live, n_next, ih_next);
      step(IC<2>{}, IC<0>{}, s + 2, next_live, next_live, n_next, ih_next);
      step(IC<3>{}, IC<1>{}, s + 3, next_live, next_live, n_next, ih_next);
      step(IC<4>{}, IC<0>{}, s + 4, next_live, next_live, n_next, ih_next);
      step(IC<5>{}, IC<1>{}, s + 5, next_live, next_live, n_next, ih_next);
    }

    // ---- epilogue, per output channel block bj and column half bc (the
    // two output rows of the tile): ops before the pool on the pre-pool
    // values, the pool in registers, ops after it on the pooled values.  The
    // bf16 results are staged in LDS, in the halo slots of this tile's input
    // rows 0 and 1 (last read in step 11), as [channel][row][pixels], a
    // 16-byte chunk q of row (co, r) at chunk q ^ (co & 15), then written out
    // with 16-byte stores, so that each store instruction covers whole
    // 128-byte lines of the output rows instead of 32 scattered channels.
    // Pooled, the whole tile (128 channels x 64 pixels) fits one slot; else
    // each channel block bj (64 channels x 2 rows x 128 pixels) fills both
    // slots and is stored before the next is staged.
    unsigned char* const slot_a = sHalo + rb * kSlot;
    unsigned char* const slot_b = sHalo + ((rb + 1) & 3) * kSlot;
    // staging row (64 channels x 2 rows of 256 bytes, unpooled)
    auto stage_row = [&](int row) { return row < 64 ? slot_a + row * 256 : slot_b + (row - 64) * 256; };
    const __amdgpu_buffer_rsrc_t ro =
        make_rsrc(out + (int64_t)n_img * COUT * plane_out, (uint32_t)(COUT * plane_out * 2));
    static_for<0, 2>([&](auto bj_c) {
      constexpr int bj = decltype(bj_c)::value;
      const int co = wn * 64 + bj * 32 + (lane & 31);
      static_for<0, 2>([&](auto bc_c) {
        constexpr int bc = decltype(bc_c)::value;
        float v[32];  // v[r * 16 + i] = acc[2 r + bc][bj][i]: output row r
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          v[i] = acc_read(acc[bc][bj][i]);
          v[16 + i] = acc_read(acc[bc + 2][bj][i]);
        }
        constexpr bool kPoolFirst = chain_pools_first(CH);
        if constexpr (!kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias_v[bj], v);
        if (p.pool) {
          // window (q, h2): columns i, i + 1 (i = 4q + 2 h2) of both rows
          float pv[8];
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
              const int i = q * 4 + h2 * 2;
              pv[q * 2 + h2] = fmaxf(fmaxf(v[i], v[i + 1]), fmaxf(v[16 + i], v[16 + i + 1]));
            }
          if constexpr (kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias_v[bj], pv);
          conv_apply_phase<CH>(ops, pidx + 1, nops, bias_v[bj], pv);
          // pooled row of channel co: 64 pixels = 8 chunks of 16 bytes
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int pw = wm * 32 + bc * 16 + q * 4 + (lane >> 5) * 2;
            const int ch = pw >> 3;
            *reinterpret_cast<uint32_t*>(slot_a + co * 128 + ((ch ^ (co & 7)) << 4) + (pw & 7) * 2) =
                pack_bf16x2(pv[q * 2], pv[q * 2 + 1]);
          }
        } else {
          const int col = wn * 32 + (lane & 31);  // channel within block bj
#pragma unroll
          for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int ow = wm * 64 + bc * 32 + q * 8 + (lane >> 5) * 4;
              const float* x = &v[r * 16 + q * 4];
              *reinterpret_cast<u32x2*>(stage_row(col * 2 + r) + (((ow >> 3) ^ (co & 15)) << 4) + (ow & 7) * 2) =
                  u32x2{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
            }
        }
      });
      if (!p.pool) {
        // channel block bj: 64 channels x 2 rows x 16 chunks
        __syncthreads();
        const uint32_t row_off = (uint32_t)(oh0 * WID * 2);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int idx = tid + 256 * k;
          const int row = idx >> 4, ch = idx & 15;
          const int col = row >> 1, r = row & 1;
          const int co = (col >> 5) * 64 + bj * 32 + (col & 31);
          const u32x4 w = *reinterpret_cast<const u32x4*>(stage_row(row) + ((ch ^ (co & 15)) << 4));
          buf_store16(w, ro, (uint32_t)(co * plane_out * 2) + row_off + (uint32_t)(r * WID * 2) + ch * 16);
        }
        __syncthreads();
      }
    });
    if (p.pool) {
      // 128 channels x 8 chunks
      __syncthreads();
      const uint32_t row_off = (uint32_t)(ph * (WID / 2) * 2);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int idx = tid + 256 * k;
        const int co = idx >> 3, ch = idx & 7;
        const u32x4 w = *reinterpret_cast<const u32x4*>(slot_a + co * 128 + ((ch ^ (co & 7)) << 4));
        buf_store16(w, ro, (uint32_t)(co * plane_out * 2) + row_off + ch * 16);
      }
    }
  }
  // nothing may land in LDS after the workgroup ends
  wait_vmcnt_lgkm0<0>();
}

// ---------------------------------------------------------------------------
// The same tile (two output rows x 128 columns x 128 channels) on 8 waves, 2 x
// 4 in (channels, pixels): each wave owns 32 columns of both rows x 64
// channels = 2 x 2 blocks of v_mfma_f32_32x32x16_bf16 (row block bi = output
// row bi), so two waves share each SIMD.  The 4-wave kernel's K-step is held
// back by its LDS reads: every CU reads 48 KiB of fragments per 512 clocks of
// matrix-core issue, and one wave per SIMD draws only ~132 bytes/clock from
// the LDS; two waves per SIMD draw ~256.  Here the CU reads 64 KiB per step
// (smaller wave blocks reuse each fragment less), half of what the LDS then
// supplies.  Halo ring, weight stream and the epilogue are the 4-wave
// kernel's, with the DMA work spread over 8 waves: one weight DMA per wave and
// step, the next tile's input rows by 4 DMAs per wave on steps 0, 2, 4 and 6;
// the 18 K-steps of a tile are unrolled, so every wait count is a constant.
namespace {

constexpr int NT8 = 512;
constexpr int kRawDma8 = kRaw / 1024 / 8;  // 4 row DMA instructions per wave per tile
static_assert(kRawDma8 == 4, "the wait counts below assume 4 row DMAs per wave, on steps 0, 2, 4, 6");

constexpr bool w8_row_step(int s) { return s >= 0 && s < 2 * kRawDma8 && s % 2 == 0; }

// Vector-memory instructions a wave issues after the weight DMA of step s - 5
// and before step s's wait: the weight DMAs of steps s-4 .. s-1 and the row
// DMAs of steps s-5 .. s-1 (steps before 0 are the previous tile's, or the
// prologue's, which issue weights only).
constexpr int w8_wait(int s) {
  int n = 4;
  for (int t = s - 5; t < s; ++t) n += w8_row_step(t) ? 1 : 0;
  return n;
}

typedef f32x16 CAcc8[2][2];

}  // namespace

template <int CH>
__global__ __launch_bounds__(NT8, 1) void kf_conv3x3_bf16_w8(ConvArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(1024))) unsigned char sHalo[kHalo];
  __shared__ __attribute__((aligned(1024))) unsigned char sRaw[kRaw];
  __shared__ __attribute__((aligned(1024))) unsigned char sW0[kWStage], sW1[kWStage], sW2[kWStage], sW3[kWStage],
      sW4[kWStage], sW5[kWStage];
  auto stW = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sW0 : S == 1 ? sW1 : S == 2 ? sW2 : S == 3 ? sW3 : S == 4 ? sW4 : sW5;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 3;   // 32-column quarter of the tile
  const int wn = wave >> 2;  // 64-channel half
  const int H = (int)p.H;
  const int rows_per_img = H / 2;
  const int64_t img_elems = (int64_t)CIN * H * WID;

  // ---- halo ring and raw rows: as in the 4-wave kernel; wave w's DMA i
  // (0 .. 3) fetches channels 2 (4 w + i) and 2 (4 w + i) + 1
  auto rsw = [](int c) { return ((c >> 3) << 1) & 15; };
  auto raw_dma = [&](int i, int n_img, int ih0, bool live) {
    const int c = 2 * (wave * kRawDma8 + i) + (lane >> 5);
    const int ih = ih0 + ((lane >> 4) & 1);
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(reinterpret_cast<const uint16_t*>(p.x) + (live ? n_img : 0) * img_elems, (uint32_t)(img_elems * 2));
    const int q = (lane & 15) ^ rsw(c);
    const bool ok = live && ih >= 0 && ih < H;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS3 void*)(sRaw + (wave * kRawDma8 + i) * 1024), 16,
                                              ok ? (uint32_t)(((c * H + ih) * WID + q * 8) * 2) : kOOB, 0, 0, 0);
  };
  // sRaw -> halo slots s0 (its row 0) and s1 (row 1), zero padding columns;
  // the first 256 threads transpose one 8 x 8 block each (spreading the
  // blocks over all 512 threads as half blocks measured slower)
  auto halo_write = [&](int s0, int s1) {
    if (tid < 256) {
      const int cg = tid & 7, pg = (tid >> 3) & 15, r = tid >> 7;
      const int slot = r ? s1 : s0;
      u32x4 hv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int c = cg * 8 + j;
        hv[j] = *reinterpret_cast<const u32x4*>(sRaw + c * 512 + r * 256 + ((pg ^ rsw(c)) << 4));
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t sel = (k & 1) ? 0x07060302u : 0x05040100u;
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = __builtin_amdgcn_perm(hv[2 * e + 1][k >> 1], hv[2 * e][k >> 1], sel);
        const int pix = slot * HALO_COLS + pg * 8 + k + 1;
        *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = o;
      }
    } else if (tid < 256 + 32) {
      const int u = tid - 256;
      const int r = u >> 4, side = (u >> 3) & 1, cg = u & 7;
      const int pix = (r ? s1 : s0) * HALO_COLS + (side ? HALO_COLS - 1 : 0);
      *reinterpret_cast<u32x4*>(sHalo + halo_off(pix, cg)) = u32x4{0u, 0u, 0u, 0u};
    }
  };

  // ---- weight stream: wave w fills rows [16 w, 16 w + 16) of a stage with
  // one DMA (chunk c of row co stored at c ^ ((co >> 2) & 3))
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)(9 * COUT * CIN * 2));
  const int dma_lc = (lane & 3) ^ ((lane >> 4) & 3);
  const uint32_t vw = (uint32_t)(((wave * 16 + (lane >> 2)) * CIN + dma_lc * 8) * 2);
  auto dma_w = [&](auto S_c, int s, bool live) {
    const int sw = s >= kSteps ? s - kSteps : s;
    const int soff = ((sw >> 1) * COUT * CIN + (sw & 1) * 32) * 2;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS3 void*)(stW(S_c) + wave * 1024), 16, live ? vw : kOOB, soff,
                                              0, 0);
  };

  // ---- fragment reads
  const int r32 = lane & 31, kg = lane >> 5;
  uint32_t rB[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int ch = kk * 2 + kg;
    rB[kk] = (uint32_t)((wn * 64 + r32) * 64 + ((ch ^ ((r32 >> 2) & 3)) << 4));
  }
  int rb = 0;                      // ring slot of logical halo row 0
  u32x4 fa[2][2][2], fb[2][2][2];  // [buffer][16-k half][block]
  constexpr int kReads8 = 8;       // per step: 4 A (2 blocks x 2 halves), 4 B
  auto read_one = [&](auto S_c, auto BUF_c, auto J_c, int s) {
    constexpr int BUF = decltype(BUF_c)::value;
    constexpr int J = decltype(J_c)::value;
    constexpr int kk = J / 4, j = J % 4;
    if constexpr (j < 2) {
      const int tap = s >> 1, kh = tap / 3, kw = tap - kh * 3;
      const int slot = (rb + j + kh) & 3;
      const int pix = slot * HALO_COLS + wm * 32 + r32 + kw;
      const int ch = (s & 1) * 4 + kk * 2 + kg;
      fa[BUF][kk][j] = lds_load<u32x4>(sHalo + halo_off(pix, ch));
    } else {
      fb[BUF][kk][j - 2] = lds_load<u32x4>(stW(S_c) + rB[kk] + (j - 2) * 2048);
    }
  };

  float bias_v[2] = {0.0f, 0.0f};
  if (p.bias) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) bias_v[bj] = p.bias[wn * 64 + bj * 32 + (lane & 31)];
  }

  CAcc8 acc;
  // K-step s (0 .. 17): wait for weight stage (s + 1) % 6 (its DMA went out
  // in step s - 5) and pass the barrier, after which every wave has read its
  // fragments of stage s % 6; then 8 MFMAs with the reads of step s + 1, the
  // weight DMA of step s + 6 into stage s % 6 and, on steps 0 .. 6 (even),
  // one DMA of the next tile's input rows.
  auto step = [&](auto s_c, bool next_live, int n_next, int ih_next) {
    constexpr int s = decltype(s_c)::value;
    constexpr int S = s % kWS, BUF = s % 2;
    wait_vmcnt_lgkm0<w8_wait(s)>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const bool live = s + kWS < kSteps || next_live;
    static_for<0, 8>([&](auto I_c) {
      constexpr int i = decltype(I_c)::value;
      constexpr int kk = i / 4, bi = (i / 2) % 2, bj = i % 2;
      acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[BUF][kk][bi]),
                                                            __builtin_bit_cast(bf16x8, fb[BUF][kk][bj]), acc[bi][bj], 0,
                                                            0, 0);
      if constexpr (s + 1 < kSteps) read_one(IC<(S + 1) % kWS>{}, IC<BUF ^ 1>{}, I_c, s + 1);
      if constexpr (i == 1) dma_w(IC<S>{}, s + kWS, live);
      if constexpr (i == 5 && w8_row_step(s)) raw_dma(s / 2, n_next, ih_next, next_live);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const int pidx = p.pool ? p.pool_index : nops;
  const int64_t plane_out = p.pool ? (int64_t)(H / 2) * (WID / 2) : (int64_t)H * WID;
  uint16_t* out = reinterpret_cast<uint16_t*>(p.out);

  const int t_begin = (int)((int64_t)blockIdx.x * p.tiles / gridDim.x);
  const int t_end = (int)((int64_t)(blockIdx.x + 1) * p.tiles / gridDim.x);
  auto continues = [&](int t) { return t > t_begin && t % rows_per_img != 0; };

  // prologue: input rows 0-1 of the first tile, then the weight stages of
  // steps 0-5, issued as K-steps -6 .. -1 would issue them (weights only)
  for (int i = 0; i < kRawDma8; ++i) raw_dma(i, t_begin / rows_per_img, 2 * (t_begin % rows_per_img) - 1, true);
  static_for<0, kWS>([&](auto S_c) { dma_w(S_c, decltype(S_c)::value, true); });

  for (int tile = t_begin; tile < t_end; ++tile) {
    const int n_img = tile / rows_per_img;
    const int ph = tile % rows_per_img;
    const int oh0 = 2 * ph;
    const bool cont = continues(tile);
    const int next_tile = tile + 1;
    const bool next_live = next_tile < t_end;
    const bool next_cont = next_live && continues(next_tile);
    const int n_next = next_tile / rows_per_img;
    const int ih_next = 2 * (next_tile % rows_per_img) + (next_cont ? 1 : -1);

    // This tile's input rows (requested in steps 0-6 of the previous tile,
    // or in the prologue) and weight stage 0 (step 12, or the prologue) have
    // landed once at most 5 vector-memory instructions are in flight: after
    // stage 0 come only the weights of steps 13-17 (prologue: of steps 1-5)
    // and the previous tile's output stores.
    wait_vmcnt_lgkm0<5>();
    __syncthreads();
    rb = cont ? (rb + 2) & 3 : 0;
    if (cont) {
      halo_write((rb + 2) & 3, (rb + 3) & 3);
    } else {
      // start of the range or of an image: rows 0-1 are in sRaw; rows 2-3
      // are requested now and waited for
      halo_write(0, 1);
      __syncthreads();
      for (int i = 0; i < kRawDma8; ++i) raw_dma(i, n_img, oh0 + 1, true);
      wait_vmcnt_lgkm0<0>();
      __syncthreads();
      halo_write(2, 3);
    }
    __syncthreads();
    static_for<0, kReads8>([&](auto J_c) { read_one(IC<0>{}, IC<0>{}, J_c, 0); });

#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int bj = 0; bj < 2; ++bj)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;

    static_for<0, kSteps>([&](auto s_c) { step(s_c, next_live, n_next, ih_next); });

    // ---- epilogue: as in the 4-wave kernel, per channel block bj, the two
    // output rows in this lane's row blocks 0 and 1
    // outputs are staged in the ring slots of this tile's input rows 0 and 1
    // (last read in step 11)
    unsigned char* const slot_a = sHalo + rb * kSlot;
    unsigned char* const slot_b = sHalo + ((rb + 1) & 3) * kSlot;
    auto stage_row = [&](int row) { return row < 64 ? slot_a + row * 256 : slot_b + (row - 64) * 256; };
    const __amdgpu_buffer_rsrc_t ro =
        make_rsrc(out + (int64_t)n_img * COUT * plane_out, (uint32_t)(COUT * plane_out * 2));
    static_for<0, 2>([&](auto bj_c) {
      constexpr int bj = decltype(bj_c)::value;
      const int co = wn * 64 + bj * 32 + (lane & 31);
      float v[32];  // v[r * 16 + i] = acc[r][bj][i]: output row r
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        v[i] = acc_read(acc[0][bj][i]);
        v[16 + i] = acc_read(acc[1][bj][i]);
      }
      constexpr bool kPoolFirst = chain_pools_first(CH);
      if constexpr (!kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias_v[bj], v);
      if (p.pool) {
        float pv[8];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int h2 = 0; h2 < 2; ++h2) {
            const int i = q * 4 + h2 * 2;
            pv[q * 2 + h2] = fmaxf(fmaxf(v[i], v[i + 1]), fmaxf(v[16 + i], v[16 + i + 1]));
          }
        if constexpr (kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias_v[bj], pv);
        conv_apply_phase<CH>(ops, pidx + 1, nops, bias_v[bj], pv);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int pw = wm * 16 + q * 4 + (lane >> 5) * 2;
          const int ch = pw >> 3;
          *reinterpret_cast<uint32_t*>(slot_a + co * 128 + ((ch ^ (co & 7)) << 4) + (pw & 7) * 2) =
              pack_bf16x2(pv[q * 2], pv[q * 2 + 1]);
        }
      } else {
        const int col = wn * 32 + (lane & 31);  // channel within block bj
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int ow = wm * 32 + q * 8 + (lane >> 5) * 4;
            const float* x = &v[r * 16 + q * 4];
            *reinterpret_cast<u32x2*>(stage_row(col * 2 + r) + (((ow >> 3) ^ (co & 15)) << 4) + (ow & 7) * 2) =
                u32x2{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
          }
        // channel block bj: 64 channels x 2 rows x 16 chunks
        __syncthreads();
        const uint32_t row_off = (uint32_t)(oh0 * WID * 2);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int idx = tid + NT8 * k;
          const int row = idx >> 4, ch = idx & 15;
          const int col2 = row >> 1, r = row & 1;
          const int co2 = (col2 >> 5) * 64 + bj * 32 + (col2 & 31);
          const u32x4 w = *reinterpret_cast<const u32x4*>(stage_row(row) + ((ch ^ (co2 & 15)) << 4));
          buf_store16(w, ro, (uint32_t)(co2 * plane_out * 2) + row_off + (uint32_t)(r * WID * 2) + ch * 16);
        }
        __syncthreads();
      }
    });
    if (p.pool) {
      // 128 channels x 8 chunks
      __syncthreads();
      const uint32_t row_off = (uint32_t)(ph * (WID / 2) * 2);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int idx = tid + NT8 * k;
        const int co = idx >> 3, ch = idx & 7;
        const u32x4 w = *reinterpret_cast<const u32x4*>(slot_a + co * 128 + ((ch ^ (co & 7)) << 4));
        buf_store16(w, ro, (uint32_t)(co * plane_out * 2) + row_off + ch * 16);
      }
    }
  }
  // nothing may land in LDS after the workgroup ends
  wait_vmcnt_lgkm0<0>();
}

// ---------------------------------------------------------------------------
// The general 3x3 convolution: any batch, cin, cout, H, W (pooling: even H
// and W).  The shapes outside the tiled kernels' family take this simpler
// implicit GEMM.  Tile: 4 output rows x 32 columns x 128 output channels per
// workgroup of 4 waves; wave w owns channels [32 w, 32 w + 32) of the tile
// and all four rows (four 32 x 32 MFMA blocks, so each weight fragment
// serves four, and a 2x2 pooling window sits in one lane's accumulators).
// k = (ci chunk of 16, tap): per chunk the input
// patch -- 6 rows x 34 columns x 16 channels, zero outside the image and past
// cin -- is staged in LDS as [pixel][16 channels] (32 bytes per pixel, so an
// A fragment is one 16-byte read), loaded into registers one chunk ahead;
// the B fragments (weights repacked to [tap][cout][cin rounded up to 16],
// zero-padded) come straight from global memory, where the whole weight set
// stays in L2.
namespace {

constexpr int kGenCols = 32, kGenRows = 4, kGenCo = 128;
constexpr int kGenPatchCols = kGenCols + 2, kGenPatchRows = kGenRows + 2;
constexpr int kGenPatch = 16 * kGenPatchRows * kGenPatchCols;  // 3264 elements per chunk
constexpr int kGenLoads = (kGenPatch + 255) / 256;              // 13 per thread

}  // namespace

__host__ __device__ int conv_gen_cin_pad(int cin) { return (cin + 15) / 16 * 16; }

// wp[tap][co][ci] = w[co][ci][kh][kw] for ci < cin, 0 up to the padded cin
__global__ __launch_bounds__(256) void kf_conv_pack_weights_gen(const uint16_t* __restrict__ w,
                                                                uint16_t* __restrict__ wp, int cout, int cin,
                                                                int cin16) {
  const int64_t pairs = (int64_t)cout * cin16;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < pairs; e += (int64_t)gridDim.x * 256) {
    const int co = (int)(e / cin16), ci = (int)(e % cin16);
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
      wp[tap * pairs + e] = ci < cin ? w[((int64_t)co * cin + ci) * 9 + tap] : (uint16_t)0;
  }
}

template <int CH>
__global__ __launch_bounds__(256) void kf_conv3x3_bf16_gen(ConvArgs p, const uint16_t* __restrict__ wp) {
  __shared__ __attribute__((aligned(16))) uint16_t sP[kGenPatch];  // [row][col][16 ci]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int H = (int)p.H, W = (int)p.W, cin = (int)p.cin, cout = (int)p.cout;
  const int cin16 = conv_gen_cin_pad(cin);
  const int chunks = cin16 / 16;
  const int tiles_co = (cout + kGenCo - 1) / kGenCo;
  const int tiles_w = (W + kGenCols - 1) / kGenCols;
  const int tiles_h = (H + kGenRows - 1) / kGenRows;
  int b = blockIdx.x;
  const int tc = b % tiles_co;
  b /= tiles_co;
  const int tw = b % tiles_w;
  b /= tiles_w;
  const int th = b % tiles_h;
  const int n = b / tiles_h;
  const int oh0 = th * kGenRows, ow0 = tw * kGenCols;
  const int co0 = tc * kGenCo + wave * 32;
  const bool wave_live = co0 < cout;  // waves past cout compute nothing (they still meet every barrier)
  const uint16_t* x = reinterpret_cast<const uint16_t*>(p.x) + (int64_t)n * cin * H * W;

  // this thread's patch elements: e = tid + 256 j -> (ci, row, col), ci fastest
  uint16_t pre[kGenLoads];
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int j = 0; j < kGenLoads; ++j) {
      const int e = tid + 256 * j;
      const int ci = e & 15, pix = e >> 4;
      const int row = pix / kGenPatchCols, col = pix % kGenPatchCols;
      const int ih = oh0 - 1 + row, iw = ow0 - 1 + col, cc = c * 16 + ci;
      pre[j] = (e < kGenPatch && cc < cin && ih >= 0 && ih < H && iw >= 0 && iw < W)
                   ? x[((int64_t)cc * H + ih) * W + iw]
                   : (uint16_t)0;
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int j = 0; j < kGenLoads; ++j) {
      const int e = tid + 256 * j;
      if (e < kGenPatch) sP[e] = pre[j];
    }
  };
  // B fragments of a chunk: lane (co0 + lane % 32, channels 8 (lane / 32) .. + 7)
  const int r32 = lane & 31, kg = lane >> 5;
  const int co_l = co0 + r32;
  const int64_t taps_stride = (int64_t)cout * cin16;
  u32x4 fb[9];
  auto load_b = [&](int c) {
#pragma unroll
    for (int tap = 0; tap < 9; ++tap)
      fb[tap] = co_l < cout ? *reinterpret_cast<const u32x4*>(wp + tap * taps_stride + (int64_t)co_l * cin16 + c * 16 +
                                                             kg * 8)
                            : u32x4{0u, 0u, 0u, 0u};
  };

  f32x16 acc[kGenRows];
#pragma unroll
  for (int r = 0; r < kGenRows; ++r)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[r][i] = 0.0f;

  load_chunk(0);
  store_chunk();
  __syncthreads();
  for (int c = 0; c < chunks; ++c) {
    if (wave_live) load_b(c);
    if (c + 1 < chunks) load_chunk(c + 1);
    if (wave_live) {
#pragma unroll
      for (int tap = 0; tap < 9; ++tap) {
        const int kh = tap / 3, kw = tap % 3;
#pragma unroll
        for (int r = 0; r < kGenRows; ++r) {
          const int pix = (r + kh) * kGenPatchCols + r32 + kw;
          const u32x4 a = *reinterpret_cast<const u32x4*>(sP + pix * 16 + kg * 8);
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                           __builtin_bit_cast(bf16x8, fb[tap]), acc[r], 0, 0, 0);
        }
      }
    }
    __syncthreads();
    if (c + 1 < chunks) {
      store_chunk();
      __syncthreads();
    }
  }
  if (!wave_live) return;

  // epilogue: acc[r][i] = output row oh0 + r, column ow0 + (i / 4) * 8 +
  // (lane / 32) * 4 + i % 4, channel co_l
  if (co_l >= cout) return;
  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const int pidx = p.pool ? p.pool_index : nops;
  const float bias = p.bias ? p.bias[co_l] : 0.0f;
  uint16_t* out = reinterpret_cast<uint16_t*>(p.out);
  // rows in pairs (0, 1) and (2, 3): a pair is one pooled row
#pragma unroll
  for (int rp = 0; rp < kGenRows / 2; ++rp) {
    float v[32];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      v[i] = acc[2 * rp][i];
      v[16 + i] = acc[2 * rp + 1][i];
    }
    constexpr bool kPoolFirst = chain_pools_first(CH);
    if constexpr (!kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias, v);
    if (p.pool) {
      const int Ho = H / 2, Wo = W / 2;
      const int ph = oh0 / 2 + rp;
      float pv[8];
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int i = q * 4 + h2 * 2;
          pv[q * 2 + h2] = fmaxf(fmaxf(v[i], v[i + 1]), fmaxf(v[16 + i], v[16 + i + 1]));
        }
      if constexpr (kPoolFirst) conv_apply_phase<CH>(ops, 0, pidx, bias, pv);
      conv_apply_phase<CH>(ops, pidx + 1, nops, bias, pv);
      if (ph < Ho) {
        uint16_t* orow = out + (((int64_t)n * cout + co_l) * Ho + ph) * Wo;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int pw = (ow0 + (q / 2) * 8 + kg * 4) / 2 + (q & 1);
          if (pw < Wo) orow[pw] = (uint16_t)f32_to_bf16_rne(pv[q]);
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int oh = oh0 + 2 * rp + r;
        if (oh >= H) continue;
        uint16_t* orow = out + (((int64_t)n * cout + co_l) * H + oh) * W;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int ow = ow0 + (i / 4) * 8 + kg * 4 + (i & 3);
          if (ow < W) orow[ow] = (uint16_t)f32_to_bf16_rne(v[r * 16 + i]);
        }
      }
    }
  }
}

hipError_t launch_conv_pack(const ConvArgs& args, void* packed_weights, hipStream_t stream) {
  if (args.variant == 2) {
    const int cin16 = conv_gen_cin_pad((int)args.cin);
    const int64_t pairs = args.cout * cin16;
    const unsigned blocks = (unsigned)((pairs + 255) / 256 < 1024 ? (pairs + 255) / 256 : 1024);
    hipLaunchKernelGGL(kf_conv_pack_weights_gen, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, stream,
                       reinterpret_cast<const uint16_t*>(args.w), reinterpret_cast<uint16_t*>(packed_weights),
                       (int)args.cout, (int)args.cin, cin16);
    return hipGetLastError();
  }
  const int64_t pairs = args.cout * args.cin;
  const unsigned blocks = (unsigned)((pairs + 255) / 256 < 1024 ? (pairs + 255) / 256 : 1024);
  hipLaunchKernelGGL(kf_conv_pack_weights, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, stream,
                     reinterpret_cast<const uint16_t*>(args.w), reinterpret_cast<uint16_t*>(packed_weights),
                     (int)args.cout, (int)args.cin);
  return hipGetLastError();
}

hipError_t launch_conv_bf16(const ConvArgs& args, const void* packed_weights, int chain, hipStream_t stream) {
  const uint16_t* wp = reinterpret_cast<const uint16_t*>(packed_weights);
  if (args.variant == 2) {
    const int64_t tiles = conv_gen_tiles(args.batch, args.H, args.W, args.cout);
    if (tiles <= 0) return hipSuccess;
    if (chain == 7)
      hipLaunchKernelGGL(kf_conv3x3_bf16_gen<7>, dim3((unsigned)tiles), dim3(256), 0, stream, args, wp);
    else
      hipLaunchKernelGGL(kf_conv3x3_bf16_gen<0>, dim3((unsigned)tiles), dim3(256), 0, stream, args, wp);
    return hipGetLastError();
  }
  if (args.tiles <= 0) return hipSuccess;
  const dim3 grid((unsigned)(args.grid < args.tiles ? args.grid : args.tiles));
  if (args.variant == 1) {
    if (chain == 7)
      hipLaunchKernelGGL(kf_conv3x3_bf16_w8<7>, grid, dim3(NT8), 0, stream, args, wp);
    else
      hipLaunchKernelGGL(kf_conv3x3_bf16_w8<0>, grid, dim3(NT8), 0, stream, args, wp);
  } else if (chain == 7) {
    hipLaunchKernelGGL(kf_conv3x3_bf16_256x128<7>, grid, dim3(NT), 0, stream, args, wp);
  } else {
    hipLaunchKernelGGL(kf_conv3x3_bf16_256x128<0>, grid, dim3(NT), 0, stream, args, wp);
  }
  return hipGetLastError();
}

int64_t conv_gen_tiles(int64_t batch, int64_t H, int64_t W, int64_t cout) {
  return batch * ((H + kGenRows - 1) / kGenRows) * ((W + kGenCols - 1) / kGenCols) * ((cout + kGenCo - 1) / kGenCo);
}

int conv_bf16_cin() { return CIN; }
int conv_bf16_width() { return WID; }
int conv_bf16_cout() { return COUT; }

}  // namespace kf
