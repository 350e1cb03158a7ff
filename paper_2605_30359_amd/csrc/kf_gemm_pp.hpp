// bf16 / fp8 GEMM + fused epilogue with 128 x 256 tiles and two workgroups
// per CU (launch variant 1 of a GEMM plan, B in [K, N] layout): the
// autotuner's second tile shape.  Every output's sum over k runs through the
// same MFMAs in the same order as in the 256x256 kernel, and the epilogue is
// the same code, so both give the same bits.
//
// The 256x256 kernel runs one workgroup per CU, so while a workgroup runs its
// epilogue (VALU work and the output / residual traffic) the matrix cores of
// its CU idle, and every CU reaches that point at the same time.  Here the
// tile is halved -- 128 x 256 outputs, 4 waves as 2 x 2, each 64 x 128 = 2 x 4
// blocks of 32 x 32 -- so that the accumulators (128 registers per lane) and
// the LDS (77 KiB) leave room for a second workgroup on the same CU.  The
// launch is persistent: two workgroups per CU walk the tiles, and the second
// of each pair starts late, so that one workgroup's epilogue overlaps the
// other's K loop on the same SIMDs.  The smaller tile needs 1.5x the LDS and
// L2 bytes per MFMA and its LDS share allows three stages, so on large GEMMs
// it is the slower shape; on short ones (a few hundred rows), where 256-row
// tiles leave CUs idle, it is the faster one.  The tuner times both.
//
//   K loop   64 bytes of k per step, three LDS stages, DMA two steps ahead;
//            each step is two phases of MFMAs, the fragments of a phase read
//            during the phase before it (one barrier per step, between the
//            phases), so only about one step of fragments is held in
//            registers: 128 accumulators + 48 (fp8: 64) fragment registers
//            fit the 256 of a wave at two waves per SIMD
//   LDS      A: [128 rows][64 B], 16-byte chunk c of row m at c ^ ((m >> 2) & 3)
//            (as in the 256x256 kernel).  B: [k][256 n] rows without padding
//            (bf16: 32 rows of 512 B, fp8: 64 rows of 256 B), chunk c of
//            k-row k at c ^ sw(k), sw(k) = 4 (k & 3) for bf16, 2 (k & 7) for
//            fp8: a 32-lane transposing read covers 4 (8) consecutive k-rows,
//            which this puts in distinct 64 (32) byte slots of the 256-byte
//            bank line
//   order    workgroup b runs on XCD b % 8; each XCD takes a contiguous eighth
//            of the tiles, rasterised in groups of 8 tile rows, so the
//            workgroups of one XCD share A rows and B columns in its L2
#pragma once

#include "kf_gemm_epilogue.hpp"


namespace kf {

namespace {

constexpr int kPpBM = 128;
constexpr int kPpDelay = 4;  // start delay of the second workgroup of a CU, in units of 8128 clocks
constexpr int kPpAStage = kPpBM * 64;  // 8 KiB
constexpr int kPpBStage = 16 * 1024;   // 16 KiB = 16 DMA blocks of 1 KiB

// Tile `i` of workgroup `b` in a persistent grid of G workgroups; false once
// the workgroup has no tile left.
__device__ __forceinline__ bool pp_tile(int b, int i, int G, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int T = tiles_m * tiles_n;
  int lid;
  if ((T & 7) == 0 && (G & 7) == 0) {
    const int per_xcd = T >> 3;
    const int local = i * (G >> 3) + (b >> 3);
    if (local >= per_xcd) return false;
    lid = (b & 7) * per_xcd + local;
  } else {
    lid = b + i * G;
    if (lid >= T) return false;
  }
  constexpr int GR = 8;
  const int per_group = GR * tiles_n;
  const int group = lid / per_group;
  const int first_m = group * GR;
  const int gsize = min(tiles_m - first_m, GR);
  const int r = lid - group * per_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
  return true;
}

}  // namespace

template <bool FP8, int EPI, int CH>
__global__ __launch_bounds__(NT, 2) void kf_gemm_mfma_pp128x256(GemmArgs p) {
  using C = ElemCfg<FP8>;
  constexpr int ES = C::ES;
  constexpr int RB = 2;
  constexpr int BMp = kPpBM;
  constexpr int kRowB = FP8 ? 256 : 512;  // bytes of one B k-row in LDS
  __shared__ __attribute__((aligned(1024))) unsigned char sA0[kPpAStage], sA1[kPpAStage], sA2[kPpAStage];
  __shared__ __attribute__((aligned(1024))) unsigned char sB0[kPpBStage], sB1[kPpBStage], sB2[kPpBStage];
  __shared__ __attribute__((aligned(16))) float sCol[3 * 256];  // bias, gamma, beta of the tile's columns
  __shared__ float sRed[2 * 256];                              // cross-wave row reductions
  auto stA = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sA0 : S == 1 ? sA1 : sA2;
  };
  auto stB = [&](auto S_c) -> unsigned char* {
    constexpr int S = decltype(S_c)::value;
    return S == 0 ? sB0 : S == 1 ? sB1 : sB2;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int K = (int)p.K;
  const int64_t lda = p.lda, ldb = p.ldb;
  const unsigned char* A = reinterpret_cast<const unsigned char*>(p.a);
  const unsigned char* B = reinterpret_cast<const unsigned char*>(p.b);
  const OpTable ops = load_op_table(p.prog, lane);
  const int nk = (K + C::KSTEP - 1) / C::KSTEP;
  const bool res_bf16 = p.residual != nullptr && p.residual_bf16;  // the residual tile goes through LDS

  // ---- loop-invariant offsets
  // A DMA: wave w fills rows [32w, 32w + 32) with 2 instructions of 16 rows;
  // lane l -> row 16i + l/4, LDS chunk l%4, holding global chunk (l%4) ^ ((l >> 4) & 3)
  const int dma_lc = (lane & 3) ^ ((lane >> 4) & 3);
  uint32_t va[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) va[i] = (uint32_t)((int64_t)(wave * 32 + i * 16 + (lane >> 2)) * lda * ES + dma_lc * 16);
  // B DMA: blocks b = wave + 4i of the 16 per stage; lane l writes stage byte
  // 1024 b + 16 l = k-row kr, LDS chunk cl, which holds global chunk cl ^ sw(kr)
  int bk_k[4], bk_c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pos = (wave + 4 * i) * 1024 + lane * 16;
    const int kr = pos / kRowB, cl = (pos % kRowB) >> 4;
    bk_k[i] = kr;
    bk_c[i] = cl ^ (FP8 ? 2 * (kr & 7) : 4 * (kr & 3));
  }
  // A fragment reads (as in the 256x256 kernel, 64 rows per wave)
  const int r32 = lane & 31, kg = lane >> 5;
  uint32_t rA[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ch = FP8 ? kg * 2 + h : h * 2 + kg;
    rA[h] = (uint32_t)((wm * 64 + r32) * 64 + ((ch ^ ((r32 >> 2) & 3)) << 4));
  }
  // B transposed reads, one base per column block bj (the k-row offset of a
  // read is an immediate).  16-lane group g = lane >> 4: k-group g >> 1,
  // column half g & 1.  bf16: read (kk, h) covers k-rows kk*16 + (g>>1)*8 +
  // h*4 + r, lane 4r + q at columns 4q .. 4q+3 of its half; fp8: read x covers
  // k-rows (g>>1)*32 + x*8 + r, lane 2r + q at columns 8q .. 8q+7.  The row's
  // swizzle depends on r only.
  uint32_t rBk[4];
  {
    const int g = lane >> 4;
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) {
      if (FP8) {
        const int r = (lane >> 1) & 7, q = lane & 1;
        rBk[bj] = (uint32_t)(((g >> 1) * 32 + r) * 256 + ((2 * ((4 * wn + bj) ^ r) + (g & 1)) << 4) + q * 8);
      } else {
        const int r = (lane >> 2) & 3, q = lane & 3;
        rBk[bj] = (uint32_t)(((g >> 1) * 8 + r) * 512 + ((16 * wn + 4 * (bj ^ r) + 2 * (g & 1) + (q >> 1)) << 4) +
                             (q & 1) * 8);
      }
    }
  }

  // The second workgroup of a CU (hardware workgroup slot 1) starts late, so
  // that the two run their epilogues at different times.
  if ((__builtin_amdgcn_s_getreg((31 << 11) | 4) >> 16) & 1) {
#pragma nounroll
    for (int i = 0; i < kPpDelay; ++i) __builtin_amdgcn_s_sleep(127);
  }

  // Fragment registers.  bf16: fa[kk][bi], ft[kk][2 bj + hh] per 16-k half
  // kk; fp8: fa[buffer][half][bi] (double-buffered over steps), ft[4 bj + x].
  u32x4 fa[FP8 ? 2 : 1][2][2];
  i32x2 ft[FP8 ? 1 : 2][FP8 ? 16 : 8];
  AccT<RB> acc;

  for (int it = 0;; ++it) {
    int tm, tn;
    if (!pp_tile(blockIdx.x, it, gridDim.x, p.tiles_m, p.tiles_n, tm, tn)) break;
    const int64_t m0 = (int64_t)tm * BMp;
    const int64_t n0 = (int64_t)tn * BN;
    const int rows_t = (int)min<int64_t>(BMp, p.M - m0);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + m0 * lda * ES, (uint32_t)(((rows_t - 1) * lda + K) * ES));
    // K = 0: B has no rows, every DMA lane is out of range
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(B + n0 * ES, K > 0 ? (uint32_t)(((K - 1) * ldb + (p.N - n0)) * ES) : 0u);
    uint32_t vbk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vbk[i] = (n0 + bk_c[i] * (16 / ES) < p.N) ? (uint32_t)((int64_t)bk_k[i] * ldb * ES + bk_c[i] * 16) : kOOB;

    // the previous tile's epilogue has finished with sCol, sRed and the stages
    __syncthreads();
    {
      const float* vec = wave == 0 ? p.bias : wave == 1 ? p.gamma : p.beta;
      if (wave < 3 && vec != nullptr) {
        const __amdgpu_buffer_rsrc_t rv = make_rsrc(vec + n0, (uint32_t)((p.N - n0) * 4));
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (LDS3 void*)(sCol + wave * 256), 16, (uint32_t)lane * 16u, 0, 0,
                                                  0);
      }
    }

    // DMA instruction j (0 .. 5) of K-step t into stage S: 2 of A, 4 of B.
    // The K-step enters as the scalar offset; the range check covers vector +
    // scalar offset, so B k-rows past K (and all lanes of the steps past the
    // end that the pipeline issues) read as zero.
    auto dma_one = [&](auto S_c, auto J_c, int t) {
      constexpr int J = decltype(J_c)::value;
      const int k0 = t * C::KSTEP;
      if constexpr (J < 2) {
        const bool kin = k0 + dma_lc * (16 / ES) < K;  // K tail of A
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (LDS3 void*)(stA(S_c) + wave * 2048 + J * 1024), 16,
                                                  kin ? va[J] : kOOB, k0 * ES, 0, 0);
      } else {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (LDS3 void*)(stB(S_c) + (wave + 4 * (J - 2)) * 1024), 16,
                                                  vbk[J - 2], (int)(k0 * ldb * ES), 0, 0);
      }
    };
    constexpr int kDma = 6;
    auto dma = [&](auto S_c, int t) { static_for<0, kDma>([&](auto J_c) { dma_one(S_c, J_c, t); }); };

    // A K-step runs in two phases of MFMAs.  bf16: phase kk is the 16-k half
    // kk (8 MFMAs: 2 row x 4 column blocks); fp8: phase q is column blocks
    // 2q, 2q+1 (4 MFMAs of 64 k).  The fragments a phase needs are read during
    // the phase before it: the "early" set of step t (bf16: half 0; fp8: A and
    // column blocks 0-1) during phase 1 of step t-1, the "late" set (bf16:
    // half 1; fp8: column blocks 2-3) during phase 0 of step t, so each
    // register is rewritten only after the MFMAs that use it have issued and
    // the wave holds just over one step of fragments.
    //   bf16 early/late: 2 A + 8 transposed B reads each
    //   fp8 early: 4 A + 8 transposed B reads; late: 8 transposed B reads
    constexpr int kEarly = FP8 ? 12 : 10, kLate = FP8 ? 8 : 10;
    auto read_b = [&](auto S_c, int slot, uint32_t base, uint32_t off) {
      (void)slot;
      if constexpr (FP8)
        return __builtin_amdgcn_ds_read_tr8_b64_v2i32((LDS3 i32x2*)(stB(S_c) + base + off));
      else
        return __builtin_bit_cast(i32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS3 i16x4*)(stB(S_c) + base + off)));
    };
    // read j of the early (LATE = 0) or late (LATE = 1) set of the step held
    // in stage S; fp8 A goes to buffer BUF
    auto read_one = [&](auto S_c, auto BUF_c, auto LATE_c, auto J_c) {
      constexpr int BUF = decltype(BUF_c)::value;
      constexpr int LATE = decltype(LATE_c)::value;
      constexpr int J = decltype(J_c)::value;
      if constexpr (!FP8) {
        constexpr int kk = LATE;
        if constexpr (J < 2) {
          fa[0][kk][J] = lds_load<u32x4>(stA(S_c) + rA[kk] + J * 2048);
        } else {
          constexpr int bj = (J - 2) / 2, hh = (J - 2) % 2;
          ft[kk][bj * 2 + hh] = read_b(S_c, 0, rBk[bj], (kk * 16 + hh * 4) * 512);
        }
      } else {
        if constexpr (!LATE && J < 4) {
          constexpr int h = J / 2, bi = J % 2;
          fa[BUF][h][bi] = lds_load<u32x4>(stA(S_c) + rA[h] + bi * 2048);
        } else {
          constexpr int jb = LATE ? J : J - 4;
          constexpr int bj = LATE * 2 + jb / 4, x = jb % 4;
          ft[0][bj * 4 + x] = read_b(S_c, 0, rBk[bj], x * 2048);
        }
      }
    };

#pragma unroll
    for (int bi = 0; bi < RB; ++bi)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;

    // MFMA i of phase PH (bf16: 8 per phase, fp8: 4) on A buffer BUF
    auto mfma_one = [&](auto BUF_c, auto PH_c, auto I_c) {
      constexpr int BUF = decltype(BUF_c)::value;
      constexpr int PH = decltype(PH_c)::value;
      constexpr int i = decltype(I_c)::value;
      if constexpr (!FP8) {
        constexpr int kk = PH, bi = i / 4, bj = i % 4;
        const bf16x8 bfr =
            __builtin_bit_cast(bf16x8, __builtin_shufflevector(ft[kk][bj * 2], ft[kk][bj * 2 + 1], 0, 1, 2, 3));
        acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr, __builtin_bit_cast(bf16x8, fa[0][kk][bi]),
                                                              acc[bi][bj], 0, 0, 0);
      } else {
        constexpr int bi = i / 2, bj = PH * 2 + i % 2;
        const i32x8 afr =
            __builtin_bit_cast(i32x8, __builtin_shufflevector(fa[BUF][0][bi], fa[BUF][1][bi], 0, 1, 2, 3, 4, 5, 6, 7));
        const auto lo = __builtin_shufflevector(ft[0][bj * 4], ft[0][bj * 4 + 1], 0, 1, 2, 3);
        const auto hi = __builtin_shufflevector(ft[0][bj * 4 + 2], ft[0][bj * 4 + 3], 0, 1, 2, 3);
        const i32x8 bfr = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[bi][bj] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bfr, afr, acc[bi][bj], 0, 0, 0, 127, 0, 127);
      }
    };

    // K-step t on stage S (= t mod 3), fp8 A buffer BUF (= t mod 2).
    //   top    wait for this step's early fragments (read during the last phase)
    //   phase0 MFMAs on the early set; read the late set from stage S; DMA of
    //          step t+2 into stage (S+2) mod 3, whose last reads (the late set
    //          of step t-1) every wave finished before step t-1's barrier
    //   mid    wait until only this step's DMA may be in flight (step t+1 has
    //          landed) and the late reads are done; barrier: stage S+1 is
    //          visible to every wave, and stage S is no longer read
    //   phase1 MFMAs on the late set; read step t+1's early set from stage S+1
    constexpr int NP = FP8 ? 4 : 8;  // MFMAs per phase
    auto step = [&](auto S_c, auto BUF_c, int t) {
      constexpr int S = decltype(S_c)::value;
      constexpr int BUF = decltype(BUF_c)::value;
      wait_vmcnt_lgkm0<kDma>();
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, NP>([&](auto I_c) {
        constexpr int i = decltype(I_c)::value;
        mfma_one(BUF_c, IC<0>{}, I_c);
        static_for<(i * kLate) / NP, ((i + 1) * kLate) / NP>(
            [&](auto J_c) { read_one(S_c, BUF_c, IC<1>{}, J_c); });
        static_for<(i * kDma) / NP, ((i + 1) * kDma) / NP>(
            [&](auto J_c) { dma_one(IC<(S + 2) % 3>{}, J_c, t + 2); });
        __builtin_amdgcn_sched_barrier(0);
      });
      wait_vmcnt_lgkm0<kDma>();
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, NP>([&](auto I_c) {
        constexpr int i = decltype(I_c)::value;
        mfma_one(BUF_c, IC<1>{}, I_c);
        static_for<(i * kEarly) / NP, ((i + 1) * kEarly) / NP>(
            [&](auto J_c) { read_one(IC<(S + 1) % 3>{}, IC<BUF ^ 1>{}, IC<0>{}, J_c); });
        __builtin_amdgcn_sched_barrier(0);
      });
    };

    dma(IC<0>{}, 0);
    dma(IC<1>{}, 1);
    wait_vmcnt_lgkm0<kDma>();  // stage 0 has landed
    __builtin_amdgcn_s_barrier();
    static_for<0, kEarly>([&](auto J_c) { read_one(IC<0>{}, IC<0>{}, IC<0>{}, J_c); });

    int t = 0;
    for (; t + 6 <= nk; t += 6) {
      step(IC<0>{}, IC<0>{}, t);
      step(IC<1>{}, IC<1>{}, t + 1);
      step(IC<2>{}, IC<0>{}, t + 2);
      step(IC<0>{}, IC<1>{}, t + 3);
      step(IC<1>{}, IC<0>{}, t + 4);
      step(IC<2>{}, IC<1>{}, t + 5);
    }
    if (t < nk) step(IC<0>{}, IC<0>{}, t);
    if (t + 1 < nk) step(IC<1>{}, IC<1>{}, t + 1);
    if (t + 2 < nk) step(IC<2>{}, IC<0>{}, t + 2);
    if (t + 3 < nk) step(IC<0>{}, IC<1>{}, t + 3);
    if (t + 4 < nk) step(IC<1>{}, IC<0>{}, t + 4);
    // the zero fills past the end may still be in flight: drain them before
    // the epilogue reuses the stage memory
    wait_vmcnt_lgkm0<0>();
    __syncthreads();

    // Residual tile (128 rows): wave w fetches row block w, blocks 0-2 into
    // sB0-sB2, block 3 into sA0 (rows 0-15) and sA1 (rows 16-31).
    // The epilogue's per-lane offsets do not change from tile to tile; an
    // opaque copy of the lane id keeps the compiler from computing them once
    // before the tile loop and holding them (in spilled registers) through
    // every K loop.
    int le = lane;
    asm volatile("" : "+v"(le));
    ResDma<RB> rd;
    rd.active = res_bf16;
    rd.wave = wave;
    rd.lane = le;
    rd.rows_r = rows_t;
    rd.n0 = n0;
    rd.N = p.N;
    rd.ldr = p.ldr;
    rd.da = wave == 0 ? sB0 : wave == 1 ? sB1 : wave == 2 ? sB2 : sA0;
    rd.db = wave == 0 ? sB0 + 8192 : wave == 1 ? sB1 + 8192 : wave == 2 ? sB2 + 8192 : sA1;
    rd.rr = make_rsrc(reinterpret_cast<const uint16_t*>(res_bf16 ? p.residual : p.a) + (res_bf16 ? m0 * p.ldr + n0 : 0),
                      res_bf16 ? (uint32_t)(((rows_t - 1) * p.ldr + (p.N - n0)) * 2) : 0u);
    const int rr = le & 31;
    auto resrow = [&](int jb) -> const unsigned char* {
      return jb == 0   ? sB0 + rr * 512
             : jb == 1 ? sB1 + rr * 512
             : jb == 2 ? sB2 + rr * 512
                       : (rr < 16 ? sA0 + rr * 512 : sA1 + (rr - 16) * 512);
    };
    EpiCtx c{le, wm, wn, wm * 64, rows_t, m0, n0, sRed, sCol, res_bf16,
             {resrow(wm * 2), resrow(wm * 2 + 1), nullptr, nullptr}, ops};
    // (stores straight from registers: c.stg stays null)
    run_epilogue<EPI, CH, FP8, RB>(p, c, acc, rd);
  }
}

// ------------------------------------------------------------ host launch

template <bool FP8, int CH>
inline void pp_launch_chain(const GemmArgs& p, dim3 grid, dim3 block, hipStream_t stream) {
  hipLaunchKernelGGL((kf_gemm_mfma_pp128x256<FP8, chain_epi(CH), CH>), grid, block, 0, stream, p);
}

template <bool FP8>
inline void pp_launch_shape(const GemmArgs& p, int epi, int chain, dim3 grid, dim3 block, hipStream_t stream) {
  switch (chain) {
    case 1: pp_launch_chain<FP8, 1>(p, grid, block, stream); return;
    case 2: pp_launch_chain<FP8, 2>(p, grid, block, stream); return;
    case 3: pp_launch_chain<FP8, 3>(p, grid, block, stream); return;
    case 4: pp_launch_chain<FP8, 4>(p, grid, block, stream); return;
    case 5: pp_launch_chain<FP8, 5>(p, grid, block, stream); return;
    case 6: pp_launch_chain<FP8, 6>(p, grid, block, stream); return;
    case 8: pp_launch_chain<FP8, 8>(p, grid, block, stream); return;
    case 14: pp_launch_chain<FP8, 14>(p, grid, block, stream); return;
    default: break;
  }
  switch (epi) {
    case kEpiGroupNorm:
      hipLaunchKernelGGL((kf_gemm_mfma_pp128x256<FP8, kEpiGroupNorm, 0>), grid, block, 0, stream, p);
      break;
    case kEpiRow:
      hipLaunchKernelGGL((kf_gemm_mfma_pp128x256<FP8, kEpiRow, 0>), grid, block, 0, stream, p);
      break;
    default:
      hipLaunchKernelGGL((kf_gemm_mfma_pp128x256<FP8, kEpiPlain, 0>), grid, block, 0, stream, p);
      break;
  }
}


}  // namespace kf
