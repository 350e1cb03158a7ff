// bf16 / fp8 GEMM + fused epilogue on gfx950 matrix cores.
//
// h = A * B with A [M,K] row-major and B either [K,N] ("KN", N
// contiguous) or [N,K] ("NK", K contiguous), fp32 accumulation, then the op
// list (bias, activations, scale, GroupNorm, residual add, row softmax /
// logsumexp partials) applied to the accumulator registers, then one store.
// This is the matmul + epilogue fusion the paper's search produces
// (Appendix A, "Operator Fusion"; Appendix C, the evolved matmul + activation
// kernel), laid out for CDNA4:
//
//   tile     256 x 256 outputs per workgroup of 4 waves (2 x 2); each wave
//            owns 128 x 128 = 4 x 4 blocks of 32 x 32 MFMA outputs
//            (v_mfma_f32_32x32x16_bf16, or for OCP fp8 e4m3 operands
//            v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales and the
//            per-tensor dequantisation applied to the accumulator), the shapes
//            that sustain the full matrix-core rate; accumulators in AGPRs
//   K loop   64 bytes of k per step, four LDS stages; operands move global -> LDS
//            by buffer_load ... lds (LDS DMA), issued three steps ahead, so no
//            VGPR stages operand data; out-of-range lanes of a DMA write zeros,
//            which pads ragged M, N and K tails without branches
//   LDS      A (and B in NK layout) as [rows][64 bytes of k] with an XOR swizzle
//            of the 16-byte chunks; B in KN layout kept as [k][256 n] with a
//            padded row pitch and read through ds_read_b64_tr_b16 / _tr_b8,
//            which transpose small blocks across each 16-lane group so every
//            lane receives consecutive k of one column
//   order    the B fragment is the MFMA "A" operand, so each lane's
//            accumulators are runs of 4 consecutive output columns of one row:
//            8-byte bf16 / 16-byte fp32 stores, lane-local row reductions
//   raster   workgroup ids are renumbered so that consecutive tiles land on
//            the same XCD (its own L2), in groups of 4 tile-rows
#pragma once

#include "kf_gemm_epilogue.hpp"

namespace kf {

namespace {

constexpr int BM = 256;

__device__ __forceinline__ void tile_coords(int bid, int tiles_m, int tiles_n, int G, bool xcd_remap, int& tm,
                                            int& tn) {
  const int nwg = tiles_m * tiles_n;
  int lid = bid;
  // Workgroups are dispatched round-robin over the 8 XCDs; renumber so that
  // each XCD receives a contiguous range of logical tiles.
  if (xcd_remap && (nwg & 7) == 0) lid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  // consecutive logical tiles walk a group of G tile rows column by column
  const int per_group = G * tiles_n;
  const int group = lid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int r = lid - group * per_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

// ---------------------------------------------------------------- main loop
//
// One __shared__ array per operand and stage (distinct objects, so the
// compiler's wait-count analysis can tell the stage being filled by LDS DMA
// from the stages being read).  An LDS DMA wave instruction writes 16 bytes
// per lane at M0 + 16 * lane; the swizzles below are therefore applied on the
// global side, by choosing which chunk each lane fetches.
//
// A K-step covers 64 bytes of k: 32 bf16 or 64 fp8.
// The LDS serves 256 bytes per clock, so a 16-byte-per-lane read is taken 16
// lanes at a time and an 8-byte one 32 lanes at a time; the layouts below
// give every such lane group 16 (32) distinct 16-byte (8-byte) bank slots.
//   A (and B-NK): [256 rows][64 bytes of k]; chunk c of row m stored at chunk
//     c ^ ((m >> 2) & 3): the 16 consecutive rows of a ds_read_b128 lane
//     group fall on 4 row positions x 4 chunk positions of a 256-byte line.
//   B-KN: [k][256 n] rows with a padded pitch (bf16: 32 rows of 576 bytes,
//     fp8: 64 rows of 288 bytes; 18 KiB either way), read through the
//     transposing ds_read_b64_tr_b16 / _b8: in each 16-lane group the lanes
//     point at 4 (8) k-rows and receive the k values of their own column.  A
//     pitch of 64 (32) bytes past 256-byte alignment puts one group's rows in
//     alternate 32 (16) byte slots and the other column half of the same
//     32-lane read in the slots between.
//
// MFMA: bf16 v_mfma_f32_32x32x16_bf16 (32 per step, two 16-k halves), fp8
// v_mfma_scale_f32_32x32x64_f8f6f4 with unit block scales (16 per step); both
// run at the full matrix-core rate and leave the same 32x32 accumulator
// layout, so the epilogue is shared.

constexpr int kAStage = BM * 64;           // 16 KiB
constexpr int kBStageKN = 18 * 1024;       // 18 KiB = 18 DMA blocks of 1 KiB
constexpr int kBStageNK = BN * 64;         // 16 KiB

}  // namespace

template <bool FP8, bool B_NK, int EPI, int CH>
__global__ __launch_bounds__(NT, 1) void kf_gemm_mfma_256x256(GemmArgs p) {
  // the shader-clock and constant-rate counters at the workgroup's start
  // (stored with the end values, and the shader clock at the end of the
  // prologue and of the K loop, when the caller asked for clock stamps)
  const long long stamp_c0 = clock64(), stamp_w0 = wall_clock64();
  using C = ElemCfg<FP8>;
  constexpr int ES = C::ES;
  constexpr int kBS = B_NK ? kBStageNK : kBStageKN;
  __shared__ __attribute__((aligned(1024))) unsigned char sA0[kAStage], sA1[kAStage], sA2[kAStage], sA3[kAStage];
  __shared__ __attribute__((aligned(1024))) unsigned char sB0[kBS], sB1[kBS], sB2[kBS], sB3[kBS];
  __shared__ __attribute__((aligned(1024))) unsigned char sDummy[B_NK ? 16 : 1024];
  __shared__ __attribute__((aligned(16))) float sCol[3 * 256];  // bias, gamma, beta of the tile's columns
  __shared__ float sRed[2 * 256];                              // cross-wave row reductions
  auto stA = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sA0 : S == 1 ? sA1 : S == 2 ? sA2 : sA3;
  };
  auto stB = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sB0 : S == 1 ? sB1 : S == 2 ? sB2 : sB3;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;

  int tm, tn;
  tile_coords(blockIdx.x, p.tiles_m, p.tiles_n, p.raster_group, p.xcd_remap != 0, tm, tn);
  const int64_t m0 = (int64_t)tm * BM;
  const int64_t n0 = (int64_t)tn * BN;
  const int K = (int)p.K;
  const int64_t lda = p.lda, ldb = p.ldb;

  // operand descriptors: based at the tile, records ending at the last valid
  // element, so rows past M / N (and past K for B-KN) read as zero
  const unsigned char* A = reinterpret_cast<const unsigned char*>(p.a);
  const unsigned char* B = reinterpret_cast<const unsigned char*>(p.b);
  const int64_t rows_a = min<int64_t>(BM, p.M - m0);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + m0 * lda * ES, (uint32_t)(((rows_a - 1) * lda + K) * ES));
  const int64_t rows_b = min<int64_t>(BN, p.N - n0);
  const __amdgpu_buffer_rsrc_t rb =
      B_NK ? make_rsrc(B + n0 * ldb * ES, (uint32_t)(((rows_b - 1) * ldb + K) * ES))
           : make_rsrc(B + n0 * ES, K > 0 ? (uint32_t)(((K - 1) * ldb + (p.N - n0)) * ES) : 0u);  // K = 0: B has no rows

  const OpTable ops = load_op_table(p.prog, lane);

  // The tile's per-column epilogue vectors (bias, gamma, beta) go to LDS with
  // one DMA instruction each (waves 0, 1, 2; columns past N read as zero),
  // ahead of the operand DMA, so they have landed long before the epilogue.
  {
    const float* vec = wave == 0 ? p.bias : wave == 1 ? p.gamma : p.beta;
    if (wave < 3 && vec != nullptr) {
      const __amdgpu_buffer_rsrc_t rv = make_rsrc(vec + n0, (uint32_t)((p.N - n0) * 4));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (LDS3 void*)(sCol + wave * 256), 16, (uint32_t)lane * 16u, 0, 0, 0);
    }
  }

  // ---- DMA source byte offsets (loop invariant; the K-step enters as soffset)
  // [rows][64 B] operands: wave w fills rows [64w, 64w + 64) with 4
  // instructions of 16 rows; lane l -> row 16i + l/4, LDS chunk l%4, which
  // holds global chunk (l%4) ^ ((l >> 4) & 3).
  const int dma_lc = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t va[4], vbn[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wave * 64 + i * 16 + (lane >> 2);
    va[i] = (uint32_t)((int64_t)row * lda * ES + dma_lc * 16);
    vbn[i] = (uint32_t)((int64_t)row * ldb * ES + dma_lc * 16);
  }
  // B-KN: 18 blocks of 1 KiB per stage, block b = wave + 4 i; byte q of the
  // stage is row q / BPITCH, byte (q % BPITCH) of the row (the pad reads as zero)
  uint32_t vbk[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    const int b = wave + 4 * i;
    const int pos = b * 1024 + lane * 16;
    const int k = pos / C::BPITCH, col = pos % C::BPITCH;
    const bool ok = b < 18 && col < 256 * ES && (n0 + col / ES < p.N);
    vbk[i] = ok ? (uint32_t)((int64_t)k * ldb * ES + col) : kOOB;
  }

  // DMA instruction j (0 .. kDma-1) of K-step t into stage S.  The K-step
  // enters as the scalar offset; the descriptor's range check applies to the
  // sum of vector and scalar offsets, so k-rows of B-KN past K (and every
  // lane of the steps past the end that the pipeline issues) read as zero.
  auto dma_one = [&](auto S_c, auto J_c, int t) {
    constexpr int J = decltype(J_c)::value;
    const int k0 = t * C::KSTEP;
    const bool kin = k0 + dma_lc * (16 / ES) < K;  // K tail of a k-contiguous operand
    if (J < 4) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (LDS3 void*)(stA(S_c) + wave * 4096 + J * 1024), 16,
                                                kin ? va[J] : kOOB, k0 * ES, 0, 0);
    } else if (B_NK) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (LDS3 void*)(stB(S_c) + wave * 4096 + (J - 4) * 1024), 16,
                                                kin ? vbn[J - 4] : kOOB, k0 * ES, 0, 0);
    } else if (J < 8) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (LDS3 void*)(stB(S_c) + wave * 1024 + (J - 4) * 4096), 16,
                                                vbk[J - 4], (int)(k0 * ldb * ES), 0, 0);
    } else {
      // blocks 16 and 17 belong to waves 0 and 1; the other waves issue the
      // same instruction out of range into a 1 KiB dummy region (out-of-range
      // DMA lanes still write zeros, so they must not target a live block),
      // which keeps the instruction stream free of branches
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (LDS3 void*)(wave < 2 ? stB(S_c) + (16 + wave) * 1024 : sDummy), 16,
                                                wave < 2 ? vbk[4] : kOOB, (int)(k0 * ldb * ES), 0, 0);
    }
  };
  constexpr int kDma = B_NK ? 8 : 9;
  auto dma = [&](auto S_c, int t) { static_for<0, kDma>([&](auto J_c) { dma_one(S_c, J_c, t); }); };

  // ---- fragment read offsets.  32x32 MFMA operand lane l: row / column
  // l & 31, k-group l >> 5.  bf16: fragment half h is the 16-k sub-step h
  // (chunk 2h + kg); fp8: the two halves are the 32 bytes of k-group kg
  // (chunks 2kg, 2kg + 1).
  const int r32 = lane & 31, kg = lane >> 5;
  uint32_t rA[2], rBn[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ch = FP8 ? kg * 2 + h : h * 2 + kg;
    rA[h] = (uint32_t)((wm * 128 + r32) * 64 + ((ch ^ ((r32 >> 2) & 3)) << 4));
    rBn[h] = (uint32_t)((wn * 128 + r32) * 64 + ((ch ^ ((r32 >> 2) & 3)) << 4));
  }
  // transposed B-KN reads, 16-lane group g = lane >> 4 (k-group g >> 1, column
  // half g & 1).  bf16: read (kk, h) gives k = kk*16 + (g>>1)*8 + h*4 + 0..3,
  // lane 4r + q points at k-row (.. + r), columns 4q .. 4q+3 of its half.
  // fp8: read h gives k = (g>>1)*32 + h*8 + 0..7, lane 2r + q points at k-row
  // (.. + r), columns 8q .. 8q+7 of its half.
  uint32_t rBk[4];
  {
    const int g = lane >> 4;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      if (FP8) {
        const int r = (lane >> 1) & 7, q = lane & 1;
        rBk[x] = (uint32_t)(((g >> 1) * 32 + x * 8 + r) * C::BPITCH + wn * 128 + (g & 1) * 16 + q * 8);
      } else {
        const int kk = x >> 1, h = x & 1, r = (lane >> 2) & 3, q = lane & 3;
        rBk[x] = (uint32_t)((kk * 16 + (g >> 1) * 8 + h * 4 + r) * C::BPITCH + (wn * 128 + (g & 1) * 16 + q * 4) * 2);
      }
    }
  }

  u32x4 fa[2][2][4], fb[2][2][4];  // [buffer][half][block]: A and B-NK fragments
  i32x2 ft[2][16];                 // [buffer][read]: B-KN transposed reads

  // Fragment read j of a K-step, in the order the next step consumes them.
  //   bf16: per 16-k half: 4 A, then B (4 x 2 transposed / 4 b128)
  //   fp8:  per half of the 32 bytes: 4 A (and 4 B-NK); B-KN: 16 transposed
  //         reads after the A halves
  constexpr int kReads = B_NK ? 16 : 24;
  auto read_one = [&](auto S_c, auto BUF_c, auto J_c) {
    constexpr int BUF = decltype(BUF_c)::value;
    constexpr int J = decltype(J_c)::value;
    if constexpr (!FP8) {
      constexpr int per = kReads / 2;
      constexpr int h = J / per, j = J % per;
      if constexpr (j < 4) {
        fa[BUF][h][j] = lds_load<u32x4>(stA(S_c) + rA[h] + j * 2048);
      } else if constexpr (B_NK) {
        fb[BUF][h][j - 4] = lds_load<u32x4>(stB(S_c) + rBn[h] + (j - 4) * 2048);
      } else {
        constexpr int bj = (j - 4) / 2, x = h * 2 + (j - 4) % 2;
        ft[BUF][(h * 4 + bj) * 2 + (j - 4) % 2] = __builtin_bit_cast(
            i32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS3 i16x4*)(stB(S_c) + rBk[x] + bj * 64)));
      }
    } else {
      if constexpr (J < 8) {
        constexpr int h = J / 4, bi = J % 4;
        fa[BUF][h][bi] = lds_load<u32x4>(stA(S_c) + rA[h] + bi * 2048);
      } else if constexpr (B_NK) {
        constexpr int h = (J - 8) / 4, bj = (J - 8) % 4;
        fb[BUF][h][bj] = lds_load<u32x4>(stB(S_c) + rBn[h] + bj * 2048);
      } else {
        constexpr int bj = (J - 8) / 4, x = (J - 8) % 4;
        ft[BUF][bj * 4 + x] =
            __builtin_amdgcn_ds_read_tr8_b64_v2i32((LDS3 i32x2*)(stB(S_c) + rBk[x] + bj * 32));
      }
    }
  };
  auto read_frags = [&](auto S_c, auto BUF_c) {
    static_for<0, kReads>([&](auto J_c) { read_one(S_c, BUF_c, J_c); });
  };

  AccT<4> acc;
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;

  // MFMA i of a K-step on fragment buffer BUF
  auto mfma_one = [&](auto BUF_c, auto I_c) {
    constexpr int BUF = decltype(BUF_c)::value;
    constexpr int i = decltype(I_c)::value;
    if constexpr (!FP8) {
      constexpr int kk = i / 16, bi = (i / 4) % 4, bj = i % 4;
      bf16x8 bfr;
      if constexpr (B_NK)
        bfr = __builtin_bit_cast(bf16x8, fb[BUF][kk][bj]);
      else
        bfr = __builtin_bit_cast(bf16x8, __builtin_shufflevector(ft[BUF][(kk * 4 + bj) * 2], ft[BUF][(kk * 4 + bj) * 2 + 1], 0, 1, 2, 3));
      acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr, __builtin_bit_cast(bf16x8, fa[BUF][kk][bi]),
                                                            acc[bi][bj], 0, 0, 0);
    } else {
      constexpr int bi = i / 4, bj = i % 4;
      const i32x8 afr = __builtin_bit_cast(i32x8, __builtin_shufflevector(fa[BUF][0][bi], fa[BUF][1][bi], 0, 1, 2, 3, 4, 5, 6, 7));
      i32x8 bfr;
      if constexpr (B_NK) {
        bfr = __builtin_bit_cast(i32x8, __builtin_shufflevector(fb[BUF][0][bj], fb[BUF][1][bj], 0, 1, 2, 3, 4, 5, 6, 7));
      } else {
        const auto lo = __builtin_shufflevector(ft[BUF][bj * 4], ft[BUF][bj * 4 + 1], 0, 1, 2, 3);
        const auto hi = __builtin_shufflevector(ft[BUF][bj * 4 + 2], ft[BUF][bj * 4 + 3], 0, 1, 2, 3);
        bfr = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
      acc[bi][bj] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bfr, afr, acc[bi][bj], 0, 0, 0, 127, 0, 127);
    }
  };

  // K-step t on stage S with fragments in buffer BUF.  The fragments of step
  // t were read from stage S during step t-1, so once every wave has passed
  // the barrier at the top of step t (each having waited for its own reads),
  // stage S is free: the DMA of step t+4 goes there, four steps ahead of its
  // use.  The same barrier publishes stage S+1 (DMA issued during step t-3),
  // whose fragments are read during this step.  The MFMAs run in a fixed
  // order with the reads spread from the start and the DMA instructions
  // evenly, so that neither the LDS queue nor the texture address FIFO backs
  // up into the wave's in-order instruction stream.  Past the last K-step the
  // DMA lanes are all out of range (zeros into a stage nobody reads) and the
  // reads read a stale stage that is never used, so nothing here is
  // conditional.
  const int nk = (K + C::KSTEP - 1) / C::KSTEP;
  const bool res_bf16 = p.residual != nullptr && p.residual_bf16;  // the residual tile goes through LDS
  const int rows_r = (int)min<int64_t>(BM, p.M - m0);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc(reinterpret_cast<const uint16_t*>(res_bf16 ? p.residual : p.a) + (res_bf16 ? m0 * p.ldr + n0 : 0),
                res_bf16 ? (uint32_t)(((rows_r - 1) * p.ldr + (p.N - n0)) * 2) : 0u);

  constexpr int NM = C::NMFMA;
  auto step = [&](auto S_c, auto BUF_c, int t) {
    constexpr int S = decltype(S_c)::value;
    constexpr int BUF = decltype(BUF_c)::value;
    wait_vmcnt_lgkm0<2 * kDma>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, NM>([&](auto I_c) {
      constexpr int i = decltype(I_c)::value;
      mfma_one(BUF_c, I_c);
      // reads j in [i*R/NM', (i+1)*R/NM') over the first NM' = min(NM, 24) MFMAs
      constexpr int NR = NM < 24 ? NM : 24;
      if constexpr (i < NR) {
        static_for<(i * kReads) / NR, ((i + 1) * kReads) / NR>(
            [&](auto J_c) { read_one(IC<(S + 1) & 3>{}, IC<BUF ^ 1>{}, J_c); });
      }
      if constexpr ((i * kDma) / NM != ((i + 1) * kDma) / NM) dma_one(S_c, IC<(i * kDma) / NM>{}, t + 4);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  dma(IC<0>{}, 0);
  dma(IC<1>{}, 1);
  dma(IC<2>{}, 2);
  dma(IC<3>{}, 3);
  wait_vmcnt_lgkm0<3 * kDma>();  // stage 0 has landed
  __builtin_amdgcn_s_barrier();
  const long long stamp_cp = clock64();  // end of the prologue
  read_frags(IC<0>{}, IC<0>{});

  int t = 0;
  for (; t + 4 <= nk; t += 4) {
    step(IC<0>{}, IC<0>{}, t);
    step(IC<1>{}, IC<1>{}, t + 1);
    step(IC<2>{}, IC<0>{}, t + 2);
    step(IC<3>{}, IC<1>{}, t + 3);
  }
  if (t < nk) step(IC<0>{}, IC<0>{}, t);
  if (t + 1 < nk) step(IC<1>{}, IC<1>{}, t + 1);
  if (t + 2 < nk) step(IC<2>{}, IC<0>{}, t + 2);
  // the zero fills past the end may still be in flight: drain them before
  // the epilogue reuses the stage memory
  wait_vmcnt_lgkm0<0>();
  __syncthreads();
  const long long stamp_ck = clock64();  // end of the K loop

  const bool res_lds = res_bf16;
  ResDma<4> rd;
  rd.active = res_lds;
  rd.wave = wave;
  rd.lane = lane;
  rd.rows_r = rows_r;
  rd.n0 = n0;
  rd.N = p.N;
  rd.ldr = p.ldr;
  rd.da = wave == 0 ? sA0 : wave == 1 ? sA1 : wave == 2 ? sA2 : sA3;
  rd.db = wave == 0 ? sB0 : wave == 1 ? sB1 : wave == 2 ? sB2 : sB3;
  rd.rr = rres;

  // row block bi of this wave is tile row block 4 wm + bi, fetched by wave
  // 2 wm + bi / 2 into its sA (first half) or sB (second half)
  const int rrow = (lane & 31) * 512;
  EpiCtx c{lane, wm, wn, wm * 128, rows_r, m0, n0, sRed, sCol, res_lds,
           {(wm ? sA2 : sA0) + rrow, (wm ? sB2 : sB0) + rrow, (wm ? sA3 : sA1) + rrow, (wm ? sB3 : sB1) + rrow}, ops};
  // with stage_out, bf16 output row blocks are staged in the same 16 KiB
  // regions; this wave stores rows 16 wn .. 16 wn + 15 of each
  if (p.stage_out) {
    c.stg[0] = (wm ? sA2 : sA0) + wn * 8192;
    c.stg[1] = (wm ? sB2 : sB0) + wn * 8192;
    c.stg[2] = (wm ? sA3 : sA1) + wn * 8192;
    c.stg[3] = (wm ? sB3 : sB1) + wn * 8192;
  }
  run_epilogue<EPI, CH, FP8, 4>(p, c, acc, rd);
  if (p.stamps != nullptr && blockIdx.x < p.stamp_cap) {
    const long long stamp_c1 = clock64(), stamp_w1 = wall_clock64();
    if (threadIdx.x == 0) {
      long long* st = p.stamps + 6 * (int64_t)blockIdx.x;
      st[0] = stamp_c0;
      st[1] = stamp_c1;
      st[2] = stamp_w0;
      st[3] = stamp_w1;
      st[4] = stamp_cp;
      st[5] = stamp_ck;
    }
  }
}

// ------------------------------------------------------------ host launch
//
// Each (FP8, B_NK) combination is instantiated by its own translation unit
// (kf_gemm_mfma_<in>_<layout>.hip), so the kernels compile in parallel.

template <bool FP8, bool B_NK, int CH>
inline void launch_chain(const GemmArgs& p, dim3 grid, dim3 block, hipStream_t stream) {
  hipLaunchKernelGGL((kf_gemm_mfma_256x256<FP8, B_NK, chain_epi(CH), CH>), grid, block, 0, stream, p);
}

template <bool FP8, bool B_NK>
inline void launch_shape(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  switch (chain) {
    case 1: launch_chain<FP8, B_NK, 1>(p, grid, block, stream); return;
    case 2: launch_chain<FP8, B_NK, 2>(p, grid, block, stream); return;
    case 3: launch_chain<FP8, B_NK, 3>(p, grid, block, stream); return;
    case 4: launch_chain<FP8, B_NK, 4>(p, grid, block, stream); return;
    case 5: launch_chain<FP8, B_NK, 5>(p, grid, block, stream); return;
    case 6: launch_chain<FP8, B_NK, 6>(p, grid, block, stream); return;
    case 8: launch_chain<FP8, B_NK, 8>(p, grid, block, stream); return;
    case 14: launch_chain<FP8, B_NK, 14>(p, grid, block, stream); return;
    default: break;
  }
  switch (epi) {
    case kEpiGroupNorm:
      hipLaunchKernelGGL((kf_gemm_mfma_256x256<FP8, B_NK, kEpiGroupNorm, 0>), grid, block, 0, stream, p);
      break;
    case kEpiRow:
      hipLaunchKernelGGL((kf_gemm_mfma_256x256<FP8, B_NK, kEpiRow, 0>), grid, block, 0, stream, p);
      break;
    default:
      hipLaunchKernelGGL((kf_gemm_mfma_256x256<FP8, B_NK, kEpiPlain, 0>), grid, block, 0, stream, p);
      break;
  }
}

void launch_gemm_bf16_kn(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
void launch_gemm_bf16_nk(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
void launch_gemm_fp8_kn(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
void launch_gemm_fp8_nk(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
// the 128x256 two-workgroups-per-CU kernel (kf_gemm_pp.hpp, B in KN layout)
void launch_gemm_pp_bf16(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
void launch_gemm_pp_fp8(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream);
int gemm_pp_tile_m();

}  // namespace kf
