// Shared pieces of the bf16 / fp8 GEMM kernels: the element types, LDS
// helpers and the fused epilogue that runs on the accumulator registers.
//
// A wave owns RB x 4 blocks of 32 x 32 outputs (RB row blocks of 32 rows,
// four column blocks of 32 columns; two waves side by side cover a
// 256-column tile row).  After the K loop the op list is applied to these
// accumulators and the result stored once.
#pragma once

#include <type_traits>

#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

#define LDS3 __attribute__((address_space(3)))

namespace {

constexpr int BN = 256;  // columns of a tile (and of a row-reduction partial)
constexpr int NT = 256;  // threads of a workgroup

template <typename T>
__device__ __forceinline__ T lds_load(const unsigned char* p) {
  return *reinterpret_cast<const T*>(p);
}

// s_waitcnt vmcnt(N) lgkmcnt(0), expcnt left alone
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0x0 << 8) | ((N >> 4) << 14));
}

// The accumulators of one wave, RB row blocks x 4 column blocks:
// acc[bi][bj][i]: output row    row_base + bi*32 + (lane & 31)
//                 output column wn*128 + bj*32 + (i/4)*8 + (lane >> 5)*4 + i%4
template <int RB>
using AccT = f32x16[RB][4];

// Whether the row reduction of compile-time chain `ch` comes right after a
// HARDTANH (whose upper bound then serves as the tile's row offset, when
// its bounds are at most kRowOffsetSpan apart).
constexpr float kRowOffsetSpan = 64.0f;
constexpr bool chain_row_after_hardtanh(int ch) {
  for (int o = 1; o < kChainLen[ch]; ++o)
    if (is_row_op(kChainOps[ch][o])) return kChainOps[ch][o - 1] == KF_OP_HARDTANH;
  return false;
}

// The row softmax / logsumexp op of a compile-time chain (0: none, or chain 0).
constexpr int chain_row_op(int ch) {
  for (int o = 0; o < kChainLen[ch]; ++o)
    if (is_row_op(kChainOps[ch][o])) return kChainOps[ch][o];
  return 0;
}

// Epilogue shape of a compile-time chain.
constexpr int chain_epi(int ch) {
  for (int o = 0; o < kChainLen[ch]; ++o) {
    if (kChainOps[ch][o] == KF_OP_GROUPNORM) return kEpiGroupNorm;
    if (is_row_op(kChainOps[ch][o])) return kEpiRow;
  }
  return kEpiPlain;
}

// -------------------------------------------------------------- epilogue
//
// The op list is run in up to two phases around its reduction op (GROUPNORM,
// ROW_SOFTMAX or ROW_LOGSUMEXP).  Each phase takes one 32-row block bi at a
// time -- its 64 values per lane in VGPRs, the rest of the tile in AGPRs --
// through all of the phase's element-wise ops, and the last phase stores.

struct EpiCtx {
  int lane, wm, wn;
  int row_base;                  // first tile row of this wave's row blocks
  int rows;                      // rows of the tile inside the output (min(tile rows, M - m0))
  int64_t m0, n0;
  float* red;                    // 2 x 256 floats of LDS for cross-wave row reductions
  const float* col;              // LDS: bias, gamma, beta of the tile's 256 columns
  bool res_lds;                  // the bf16 residual tile sits in LDS (see the kernel's residual staging)
  const unsigned char* res[4];   // LDS: this lane's residual row (lane & 31) of row block bi
  OpTable ops;                   // the op program, one op per lane
  // LDS staging of a bf16 output row block bi in the residual's rows (res[bi]
  // is this lane's row there): the first of the 16 rows (16 wn .. 16 wn + 15
  // of the block, 512 bytes apart) that this wave stores from LDS, or null:
  // the row block is stored from registers
  const unsigned char* stg[4];
};

// run g (0..15) of a row = block bj = g / 4, group gi = g % 4: columns
// col_local(c, 0) + run_offset(g) + 0..3
constexpr int run_offset(int g) { return (g >> 2) * 32 + (g & 3) * 8; }
__device__ __forceinline__ int col_local(const EpiCtx& c, int g) {
  return c.wn * 128 + run_offset(g) + (c.lane >> 5) * 4;
}
__device__ __forceinline__ int row_local(const EpiCtx& c, int bi) { return c.row_base + bi * 32 + (c.lane & 31); }

typedef f32x4 Row[16];  // one lane's 64 values of one row

template <int RB>
__device__ __forceinline__ void get_row(const AccT<RB>& acc, int bi, Row& v) {
#pragma unroll
  for (int g = 0; g < 16; ++g) {
    const f32x16& a = acc[bi][g >> 2];
    const int o = (g & 3) * 4;
    v[g] = f32x4{acc_read(a[o]), acc_read(a[o + 1]), acc_read(a[o + 2]), acc_read(a[o + 3])};
  }
}
template <int RB>
__device__ __forceinline__ void put_row(AccT<RB>& acc, int bi, const Row& v) {
#pragma unroll
  for (int g = 0; g < 16; ++g) {
    const int o = (g & 3) * 4;
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[bi][g >> 2][o + q] = v[g][q];
  }
}

// 4 consecutive fp32 of a per-column vector (0 bias, 1 gamma, 2 beta), staged
// in LDS at kernel start; columns >= N read as 0.
__device__ __forceinline__ f32x4 col4(const EpiCtx& c, int which, int g) {
  return *reinterpret_cast<const f32x4*>(c.col + which * 256 + col_local(c, g));
}

// The bf16 residual tile in LDS: 512 bytes per tile row, the 16-byte chunk q
// of row m stored at chunk q ^ (m & 15); where each row sits is up to the
// kernel (c.res).
__device__ __forceinline__ f32x4 res4(const EpiCtx& c, int bi, int g) {
  const int r = c.lane & 31;
  const int q = c.wn * 16 + (g >> 2) * 4 + (g & 3);
  const u32x2 w = *reinterpret_cast<const u32x2*>(c.res[bi] + ((q ^ (r & 15)) << 4) + (c.lane >> 5) * 8);
  return f32x4{bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
}

// Wait until every wave's share of the residual tile has landed in LDS.
__device__ __forceinline__ void res_wait(const EpiCtx& c) {
  if (c.res_lds) {
    wait_vmcnt_lgkm0<0>();
    __syncthreads();
  }
}

__device__ __forceinline__ float sum4(f32x4 a) { return (a[0] + a[1]) + (a[2] + a[3]); }
__device__ __forceinline__ float max4(f32x4 a) { return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3])); }

// Combine one value per row over the two lanes of the row (lane ^ 32) and, if
// `cross`, over the two waves that share the rows (through LDS).  Every
// thread of the workgroup must call it with the same `cross`.
template <bool IS_MAX, int RB>
__device__ __forceinline__ void row_combine(const EpiCtx& c, float (&v)[RB], bool cross) {
#pragma unroll
  for (int bi = 0; bi < RB; ++bi) {
    const float y = shfl_xor(v[bi], 32);
    v[bi] = IS_MAX ? fmaxf(v[bi], y) : v[bi] + y;
  }
  if (!cross) return;
  if (c.lane < 32) {
#pragma unroll
    for (int bi = 0; bi < RB; ++bi) c.red[c.wn * 256 + row_local(c, bi)] = v[bi];
  }
  __syncthreads();
#pragma unroll
  for (int bi = 0; bi < RB; ++bi) {
    const float o = c.red[(c.wn ^ 1) * 256 + row_local(c, bi)];
    v[bi] = IS_MAX ? fmaxf(v[bi], o) : v[bi] + o;
  }
  __syncthreads();
}

// Epilogue-internal op kind: a GELU_ERF whose input is the output of a TANH
// (the op before it in the list), so in [-1, 1].
constexpr int kOpGeluErfUnit = 1000;
__host__ __device__ constexpr int epi_kind(int kind, int prev) {
  return kind == KF_OP_GELU_ERF && prev == KF_OP_TANH ? kOpGeluErfUnit : kind;
}

// One element-wise / tensor-reading op (kind, at position o of the list) on
// one row block.  With a compile-time kind the switch folds away.
__device__ __forceinline__ void apply_op(const GemmArgs& p, const EpiCtx& c, int bi, int kind, int o, Row& v) {
  const int64_t N = p.N;
  {
    const float p0 = op_p0(c.ops, o), p1 = op_p1(c.ops, o);
    switch (kind) {
      case KF_OP_BIAS:
#pragma unroll
        for (int g = 0; g < 16; ++g) v[g] += col4(c, 0, g);
        break;
      case KF_OP_RESIDUAL_ADD: {
        const int64_t rows = c.rows;
        const int64_t rl = row_local(c, bi);
        if (c.res_lds) {
#pragma unroll
          for (int g = 0; g < 16; ++g) v[g] += res4(c, bi, g);
        } else if (p.residual_bf16) {
          const uint16_t* base = reinterpret_cast<const uint16_t*>(p.residual) + c.m0 * p.ldr + c.n0;
          const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldr + (N - c.n0)) * 2));
#pragma unroll
          for (int g = 0; g < 16; ++g) {
            const int cl = col_local(c, g);
            const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldr + cl) * 2) : kOOB;
            const u32x2 w = buf_load8(r, off);
            v[g] += f32x4{bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
          }
        } else {
          const float* base = reinterpret_cast<const float*>(p.residual) + c.m0 * p.ldr + c.n0;
          const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldr + (N - c.n0)) * 4));
#pragma unroll
          for (int g = 0; g < 16; ++g) {
            const int cl = col_local(c, g);
            const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldr + cl) * 4) : kOOB;
            v[g] += __builtin_bit_cast(f32x4, buf_load16(r, off));
          }
        }
        break;
      }
#define KF_EW_CASE(K, EXPR)                          \
  case K:                                            \
    _Pragma("unroll") for (int g = 0; g < 16; ++g)   \
    _Pragma("unroll") for (int q = 0; q < 4; ++q) {  \
      const float x = v[g][q];                       \
      v[g][q] = (EXPR);                              \
    }                                                \
    break;
      KF_EW_CASE(KF_OP_RELU, fmaxf(x, 0.0f))
      KF_EW_CASE(KF_OP_GELU_TANH, f_gelu_tanh(x))
      KF_EW_CASE(KF_OP_GELU_ERF, f_gelu_erf(x))
      KF_EW_CASE(kOpGeluErfUnit, f_gelu_erf_unit(x))
      KF_EW_CASE(KF_OP_SWISH, f_swish(x))
      KF_EW_CASE(KF_OP_SIGMOID, f_sigmoid(x))
      KF_EW_CASE(KF_OP_TANH, f_tanh(x))
      KF_EW_CASE(KF_OP_HARDTANH, fminf(fmaxf(x, p0), p1))
      KF_EW_CASE(KF_OP_SCALE, x * p0)
#undef KF_EW_CASE
      default:
        break;
    }
  }
}

// Ops oi..oe-1 of chain CH on one row block: interpreted (chain 0), or
// unrolled over the chain's compile-time op kinds.  Either way a GELU_ERF
// right after a TANH takes the bounded-input form (the same bits).
template <int CH>
__device__ __forceinline__ void apply_phase(const GemmArgs& p, const EpiCtx& c, int bi, int oi, int oe, Row& v) {
  if constexpr (CH == 0) {
#pragma nounroll
    for (int o = oi; o < oe; ++o) apply_op(p, c, bi, epi_kind(op_kind(c.ops, o), o > 0 ? op_kind(c.ops, o - 1) : 0), o, v);
  } else {
    static_for<0, kChainLen[CH]>([&](auto O_c) {
      constexpr int o = decltype(O_c)::value;
      constexpr int kind = epi_kind(kChainOps[CH][o], o > 0 ? kChainOps[CH][o > 0 ? o - 1 : 0] : 0);
      if (o >= oi && o < oe) apply_op(p, c, bi, kind, o, v);
    });
  }
}

// Store one row block (16 runs of 4 values per lane).  A bf16 row block
// with LDS staging goes through LDS: each lane writes its 16 runs of 8 bytes
// to its row there (the layout of the residual rows: 16-byte chunk q of row
// m at q ^ (m & 15), whose two 8-byte halves are swapped in rows 16-31, so
// that the 32 rows of one write instruction meet 32 distinct 8-byte bank
// slots; a lane overwrites only residual chunks its own wave has read),
// then, after a barrier, the two waves that share the 32 rows store 16 rows
// each, 16 bytes per lane: every store instruction writes two whole 512-byte
// tile rows, where the direct stores write 16-byte pieces of 32 rows.
// Every wave of the workgroup must call it for the same row blocks.
__device__ __forceinline__ void store_row(const GemmArgs& p, const EpiCtx& c, int bi, const Row& v) {
  const int64_t N = p.N;
  const int64_t rows = c.rows;
  const int64_t rl = row_local(c, bi);
  if (p.out_bf16 && c.stg[bi] != nullptr) {
    const int rr = c.lane & 31;
    unsigned char* own = const_cast<unsigned char*>(c.res[bi]) + (((c.lane >> 5) ^ (rr >> 4)) * 8);
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      const int q = c.wn * 16 + (g >> 2) * 4 + (g & 3);
      *reinterpret_cast<u32x2*>(own + ((q ^ (rr & 15)) << 4)) =
          u32x2{pack_bf16x2(v[g][0], v[g][1]), pack_bf16x2(v[g][2], v[g][3])};
    }
    __syncthreads();
    uint16_t* base = reinterpret_cast<uint16_t*>(p.out) + c.m0 * p.ldo + c.n0;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldo + (N - c.n0)) * 2));
    const unsigned char* half = c.stg[bi];
    const int q = c.lane & 31;
    const bool col_ok = c.n0 + q * 8 < N;
    const int64_t row0 = c.row_base + bi * 32 + c.wn * 16;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int hr = 2 * i + (c.lane >> 5);  // row within the wave's 16
      u32x4 w = *reinterpret_cast<const u32x4*>(half + hr * 512 + ((q ^ ((c.wn * 16 + hr) & 15)) << 4));
      if (c.wn) w = u32x4{w[2], w[3], w[0], w[1]};  // rows 16-31: halves swapped in LDS
      buf_store16(w, r, col_ok ? (uint32_t)(((row0 + hr) * p.ldo + q * 8) * 2) : kOOB);
    }
    return;
  }
  // Rows past M fall outside the descriptor's range.  Columns past N exist
  // only in the last column tile; in every other tile the 16 runs of a row
  // sit at fixed distances from the first, which become immediate offsets.
  const bool full = c.n0 + BN <= N;
  const int cl0 = col_local(c, 0);
  if (p.out_bf16) {
    uint16_t* base = reinterpret_cast<uint16_t*>(p.out) + c.m0 * p.ldo + c.n0;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldo + (N - c.n0)) * 2));
    u32x2 w[16];
#pragma unroll
    for (int g = 0; g < 16; ++g) w[g] = u32x2{pack_bf16x2(v[g][0], v[g][1]), pack_bf16x2(v[g][2], v[g][3])};
    if (full) {
      const uint32_t off0 = (uint32_t)((rl * p.ldo + cl0) * 2);
#pragma unroll
      for (int g = 0; g < 16; ++g) buf_store8(w[g], r, off0 + (uint32_t)(run_offset(g) * 2));
    } else {
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int cl = col_local(c, g);
        buf_store8(w[g], r, (c.n0 + cl < N) ? (uint32_t)((rl * p.ldo + cl) * 2) : kOOB);
      }
    }
  } else {
    float* base = reinterpret_cast<float*>(p.out) + c.m0 * p.ldo + c.n0;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldo + (N - c.n0)) * 4));
    if (full) {
      const uint32_t off0 = (uint32_t)((rl * p.ldo + cl0) * 4);
#pragma unroll
      for (int g = 0; g < 16; ++g)
        buf_store16(__builtin_bit_cast(u32x4, v[g]), r, off0 + (uint32_t)(run_offset(g) * 4));
    } else {
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int cl = col_local(c, g);
        buf_store16(__builtin_bit_cast(u32x4, v[g]), r, (c.n0 + cl < N) ? (uint32_t)((rl * p.ldo + cl) * 4) : kOOB);
      }
    }
  }
}

// The bf16 residual tile (RB * 64 rows x 256 columns) moves into the free
// stage memory by LDS DMA during the epilogue: wave w fetches the RB * 16
// tile rows [w * RB * 16, (w + 1) * RB * 16), the first half of them to `da`
// and the second half to `db`, 512 bytes per row, the 16-byte chunk q of row
// m at chunk q ^ (m & 15) (so the epilogue's 32-lane column reads spread over
// 16 chunk slots); one DMA instruction moves two rows, 8 * RB per wave.  The
// instructions are issued in groups between epilogue computations that do
// not need the residual: when workgroups reach this point together the burst
// is bound by HBM bandwidth, and a wave that issued them back to back would
// stall on the full address queue instead of computing.
template <int RB>
struct ResDma {
  static constexpr int kRows = RB * 16;  // tile rows fetched by one wave
  static constexpr int kInstr = kRows / 2;
  __amdgpu_buffer_rsrc_t rr;
  unsigned char* da;
  unsigned char* db;
  int wave, lane, rows_r;
  int64_t n0, N, ldr;
  bool active;
  template <int J0, int J1>
  __device__ __forceinline__ void issue() const {
    if (!active) return;
    static_for<J0, J1>([&](auto J_c) {
      constexpr int j = decltype(J_c)::value;
      const int m = wave * kRows + 2 * j + (lane >> 5);
      const int q = (lane & 31) ^ (m & 15);
      const bool ok = m < rows_r && n0 + q * 8 < N;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rr, (LDS3 void*)((j < kInstr / 2 ? da : db) + ((2 * j) & (kRows / 2 - 1)) * 512), 16,
          ok ? (uint32_t)((m * ldr + q * 8) * 2) : kOOB, 0, 0, 0);
    });
  }
};

// Epilogue of shape EPI (see EpiShape): ops [0, r) element-wise, op r the
// reduction (if any), ops (r, n) element-wise, then the store.
template <int EPI, int CH, bool FP8, int RB>
__device__ __forceinline__ void run_epilogue(const GemmArgs& p, const EpiCtx& c, AccT<RB>& acc, const ResDma<RB>& rd) {
  constexpr int kRes = ResDma<RB>::kInstr;  // residual DMA instructions per wave
  static_assert(kRes == 8 * RB, "the GroupNorm passes issue 4 residual DMAs per row block each");
  const int64_t N = p.N;
  const int nops = p.prog.n;
  const int r = EPI == kEpiPlain ? nops : p.red_index;

  if (EPI == kEpiPlain) {
    rd.template issue<0, kRes>();
    res_wait(c);
    static_for<0, RB>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      Row v;
      get_row(acc, bi, v);
#pragma unroll
      for (int g = 0; g < 16; ++g) v[g] *= FP8 ? p.scale : 1.0f;  // the bf16 path skips the multiply
      apply_phase<CH>(p, c, bi, 0, nops, v);
      store_row(p, c, bi, v);
      __builtin_amdgcn_sched_barrier(0);  // one row block's values at a time
    });
    return;
  }

  if (EPI == kEpiGroupNorm) {
    // Group width gw in {32, 64, 128, 256} columns: each lane holds 16 of
    // every 32-column block of its rows, so per-block sums are lane-local plus
    // one exchange with lane ^ 32; wider groups add neighbouring blocks, and a
    // 256-wide group also the other wave's half of the tile row.
    int res_at = -1;
    for (int o = 0; o < nops; ++o)
      if (op_kind(c.ops, o) == KF_OP_RESIDUAL_ADD) res_at = o;
    const bool res_early = res_at < r;  // the residual is added before the statistics
    if (res_early) {
      rd.template issue<0, kRes>();
      res_wait(c);
    }
    const int gw = p.gn_group;
    const int bpg = gw >> 5;  // 32-column blocks per group (1, 2, 4, 8)
    const int bw = min(bpg, 4);
    const float inv_n = 1.0f / (float)gw;
    float s[RB][4];
    // A bf16 chain that starts with the GroupNorm sums the accumulators as
    // they are (the dequantisation factor is 1), in the same order as below.
    constexpr bool kSumAcc = !FP8 && CH != 0 && kChainOps[CH][0] == KF_OP_GROUPNORM;
    static_for<0, RB>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      if (!res_early) rd.template issue<4 * bi, 4 * bi + 4>();
      if constexpr (kSumAcc) {
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) {
          const f32x16& a = acc[bi][bj];
          auto s4 = [&](int o) {
            return (acc_read(a[o]) + acc_read(a[o + 1])) + (acc_read(a[o + 2]) + acc_read(a[o + 3]));
          };
          s[bi][bj] = (s4(0) + s4(4)) + (s4(8) + s4(12));
        }
      } else {
        Row v;
        get_row(acc, bi, v);
#pragma unroll
        for (int g = 0; g < 16; ++g) v[g] *= FP8 ? p.scale : 1.0f;  // the bf16 path skips the multiply
        apply_phase<CH>(p, c, bi, 0, r, v);
#pragma unroll
        for (int bj = 0; bj < 4; ++bj)
          s[bi][bj] = (sum4(v[bj * 4]) + sum4(v[bj * 4 + 1])) + (sum4(v[bj * 4 + 2]) + sum4(v[bj * 4 + 3]));
        put_row(acc, bi, v);
      }
    });
    auto group_reduce = [&](float (&t)[RB][4]) {
#pragma unroll
      for (int bi = 0; bi < RB; ++bi)
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) t[bi][bj] += shfl_xor(t[bi][bj], 32);
#pragma unroll
      for (int bi = 0; bi < RB; ++bi) {
        float g2[4];
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) {
          float a = 0.0f;
#pragma unroll
          for (int q = 0; q < 4; ++q) a += ((q / bw) == (bj / bw)) ? t[bi][q] : 0.0f;
          g2[bj] = a;
        }
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) t[bi][bj] = g2[bj];
      }
      if (bpg == 8) {
        float w[RB];
#pragma unroll
        for (int bi = 0; bi < RB; ++bi) w[bi] = t[bi][0];
        if (c.lane < 32) {
#pragma unroll
          for (int bi = 0; bi < RB; ++bi) c.red[c.wn * 256 + row_local(c, bi)] = w[bi];
        }
        __syncthreads();
#pragma unroll
        for (int bi = 0; bi < RB; ++bi) {
          const float o = w[bi] + c.red[(c.wn ^ 1) * 256 + row_local(c, bi)];
#pragma unroll
          for (int bj = 0; bj < 4; ++bj) t[bi][bj] = o;
        }
        __syncthreads();
      }
    };
    group_reduce(s);
    float mean[RB][4], ss[RB][4];
    static_for<0, RB>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      if (!res_early) rd.template issue<kRes / 2 + 4 * bi, kRes / 2 + 4 * bi + 4>();
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) {
        mean[bi][bj] = s[bi][bj] * inv_n;
        float a = 0.0f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const float d = acc_read(acc[bi][bj][q]) - mean[bi][bj];
          a += d * d;
        }
        ss[bi][bj] = a;
      }
    });
    group_reduce(ss);
    const float eps = op_p0(c.ops, r);
    if (!res_early) res_wait(c);
    static_for<0, RB>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      Row v;
      get_row(acc, bi, v);
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int bj = g >> 2;
        const float rs = rsqrtf(ss[bi][bj] * inv_n + eps);
        const f32x4 gm = col4(c, 1, g), bt = col4(c, 2, g);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[g][q] = fmaf((v[g][q] - mean[bi][bj]) * rs, gm[q], bt[q]);
      }
      apply_phase<CH>(p, c, bi, r + 1, nops, v);
      store_row(p, c, bi, v);
    });
    return;
  }

  // kEpiRow: the tile's row offset mu (normally the tile-row max), then the
  // sum of e^(h - mu); the (mu, sum) pair of this 256-column tile goes to the
  // partials buffer, and softmax stores e^(h - mu).  Any offset gives the
  // same softmax and logsumexp after the finishing kernel (it rescales by
  // e^(mu_t - max_t mu_t) / S); the max only keeps e^(h - mu) from
  // overflowing.  When the op right before the row op is a HARDTANH with
  // bounds (lo, hi), hi - lo <= 64, every h is at most hi and e^(h - hi) is at
  // least e^-64: hi is a safe offset, and the tile takes one pass over its
  // accumulators with no max and no cross-wave max exchange.
  const int row_op = chain_row_op(CH) ? chain_row_op(CH) : op_kind(c.ops, r);
  const bool ce = row_op == KF_OP_ROW_CROSS_ENTROPY;
  const bool softmax = row_op == KF_OP_ROW_SOFTMAX;
  rd.template issue<0, kRes>();
  res_wait(c);
  // (a compiled chain with that shape is only planned when the bounds
  // qualify, so there the choice is made at compile time)
  const bool bounded = chain_row_after_hardtanh(CH) ||
                       (CH == 0 && r > 0 && op_kind(c.ops, r - 1) == KF_OP_HARDTANH &&
                        op_p1(c.ops, r - 1) - op_p0(c.ops, r - 1) <= kRowOffsetSpan);
  // the ops before the row op on one row block; columns past N become -inf
  auto prep = [&](auto bi_c, Row& v) {
    constexpr int bi = decltype(bi_c)::value;
    get_row(acc, bi, v);
#pragma unroll
    for (int g = 0; g < 16; ++g) v[g] *= FP8 ? p.scale : 1.0f;  // the bf16 path skips the multiply
    apply_phase<CH>(p, c, bi, 0, r, v);
    if (ce) {
      // cross-entropy: the one lane of the grid that holds h[m][t_m] leaves it
      // for the finishing kernel.  This lane's columns are col_local(c, g) +
      // q = wn * 128 + 32 (g / 4) + 8 (g % 4) + 4 (lane / 32) + q.
      const int64_t m = c.m0 + row_local(c, bi);
      if (m < p.M) {
        const int64_t t = p.targets[m];
        const int64_t d = t - c.n0 - c.wn * 128 - (c.lane >> 5) * 4;
        if (t < N && d >= 0 && d < 128 && (d & 4) == 0) {
          const int sel = (int)(((d >> 5) * 4 + ((d >> 3) & 3)) * 4 + (d & 3));
          float h = 0.0f;
#pragma unroll
          for (int g = 0; g < 16; ++g)
#pragma unroll
            for (int q = 0; q < 4; ++q) h = sel == g * 4 + q ? v[g][q] : h;
          p.tlogit[m] = h;
        }
      }
    }
    // columns past N take no part in a row reduction (only the last column
    // tile can have any)
    if (c.n0 + BN > N) {
#pragma unroll
      for (int g = 0; g < 16; ++g) {
        const int64_t n = c.n0 + col_local(c, g);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[g][q] = (n + q < N) ? v[g][q] : -INFINITY;
      }
    }
  };
  // e^(h - mu) of one row block in place and its sum (in the order of the
  // accumulators: block bj, element q); softmax stores the values as soon as
  // they are computed (the store needs mu, not the sum), so the output
  // traffic overlaps the remaining row blocks' work.
  auto exp_store = [&](auto bi_c, Row& v, float mu) {
    constexpr int bi = decltype(bi_c)::value;
    const float ml = mu * kLog2e;
#pragma unroll
    for (int g = 0; g < 16; ++g)
#pragma unroll
      for (int k = 0; k < 4; ++k) v[g][k] = __builtin_amdgcn_exp2f(fmaf(v[g][k], kLog2e, -ml));
    float s = 0.0f;
#pragma unroll
    for (int q = 0; q < 16; ++q)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) s += v[bj * 4 + (q >> 2)][q & 3];
    if (softmax) store_row(p, c, bi, v);
    return s;
  };
  float mx[RB], se[RB];
  const float hi = bounded ? op_p1(c.ops, r - 1) : 0.0f;
  if (!bounded) {
    static_for<0, RB>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      Row v;
      prep(bi_c, v);
      float m = -INFINITY;
#pragma unroll
      for (int g = 0; g < 16; ++g) m = fmaxf(m, max4(v[g]));
      mx[bi] = m;
      put_row(acc, bi, v);
    });
    row_combine<true>(c, mx, true);
  }
  static_for<0, RB>([&](auto bi_c) {
    constexpr int bi = decltype(bi_c)::value;
    Row v;
    if (bounded) {
      prep(bi_c, v);
      mx[bi] = hi;
    } else {
      get_row(acc, bi, v);
    }
    se[bi] = exp_store(bi_c, v, mx[bi]);
  });
  row_combine<false>(c, se, true);
  if (c.lane < 32 && c.wn == 0) {
    float2* part = reinterpret_cast<float2*>(p.partials);
    const int tn = (int)(c.n0 / BN);
#pragma unroll
    for (int bi = 0; bi < RB; ++bi) {
      const int64_t m = c.m0 + row_local(c, bi);
      if (m < p.M) part[m * p.tiles_n + tn] = make_float2(mx[bi], se[bi]);
    }
  }
}


template <bool FP8>
struct ElemCfg;
template <>
struct ElemCfg<false> {  // bf16
  static constexpr int ES = 2, KSTEP = 32, NMFMA = 32, BPITCH = 576;
};
template <>
struct ElemCfg<true> {  // OCP fp8 e4m3
  static constexpr int ES = 1, KSTEP = 64, NMFMA = 16, BPITCH = 288;
};

typedef __attribute__((ext_vector_type(4))) short i16x4;
typedef __attribute__((ext_vector_type(2))) int i32x2;

template <int V>
using IC = std::integral_constant<int, V>;

}  // namespace

}  // namespace kf
