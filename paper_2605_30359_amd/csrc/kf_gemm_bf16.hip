// bf16 GEMM + fused epilogue on gfx950 matrix cores.
//
// h = A * B with A [M,K] bf16 row-major and B either [K,N] ("KN", N
// contiguous) or [N,K] ("NK", K contiguous), fp32 accumulation, then the
// op list (bias, activations, scale, GroupNorm, residual add, row softmax /
// logsumexp partials) on the accumulator registers, then one store.  This is
// the matmul + epilogue fusion the paper's search produces (Appendix A,
// "Operator Fusion"; Appendix C, the evolved matmul + activation kernel),
// laid out for CDNA4:
//
//   tile        256 x 256 output per workgroup, BK = 64, 4 waves (2 x 2),
//               each wave 128 x 128 = 8 x 8 blocks of v_mfma_f32_16x16x32_bf16
//   operands    128-bit buffer loads (out-of-range lanes read 0: ragged M,
//               N, K need no branches), staged in registers one K-step ahead
//   LDS         two stages x (A 32 KB + B 32 KB), rows of 64 k (128 B) with
//               the 16-byte chunk index XOR-swizzled by (row & 7) so both
//               the staging writes and the fragment reads are conflict-free;
//               a KN operand is transposed 8x8 in registers (v_perm_b32)
//               while it is staged, so both operands are k-contiguous in LDS
//   MFMA order  the B fragment is passed as the MFMA "A" operand, so each
//               lane's 4 accumulator values are 4 consecutive output
//               columns of one row: 8-byte bf16 / 16-byte fp32 stores and
//               row reductions that are lane-local first
//   raster      workgroups are renumbered so that consecutive tiles land on
//               the same XCD (its own L2), in groups of 4 tile-rows
#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int BK = 64;
constexpr int NT = 256;
constexpr int kStageBytes = (BM + BN) * BK * 2;  // 64 KiB
constexpr int kOffB = BM * BK * 2;               // B follows A in a stage

// Byte offset of 16-byte chunk `chunk` (0..7) of row `row` in an LDS operand
// tile whose rows hold 64 bf16.
__device__ __forceinline__ uint32_t swz(int row, int chunk) {
  return (uint32_t)(row * 128 + ((chunk ^ (row & 7)) << 4));
}

__device__ __forceinline__ void tile_coords(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  int lid = bid;
  // Workgroups are dispatched round-robin over the 8 XCDs; renumber so that
  // each XCD receives a contiguous range of logical tiles.
  if ((nwg & 7) == 0) lid = (bid & 7) * (nwg >> 3) + (bid >> 3);
  constexpr int G = 4;
  const int per_group = G * tiles_n;
  const int group = lid / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int r = lid - group * per_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

template <typename T>
__device__ __forceinline__ T lds_load(const unsigned char* p) {
  return *reinterpret_cast<const T*>(p);
}
template <typename T>
__device__ __forceinline__ void lds_store(unsigned char* p, T v) {
  *reinterpret_cast<T*>(p) = v;
}

typedef f32x4 Acc[8][8];

// -------------------------------------------------------------- epilogue
//
// Accumulator element (bi, bj, r) of lane `lane` in wave (wm, wn) holds
// output row  m0 + wm*128 + bi*16 + (lane & 15)
// and column  n0 + wn*128 + bj*16 + (lane >> 4)*4 + r.
//
// The op list is executed in phases separated by its reduction ops
// (GROUPNORM, ROW_SOFTMAX, ROW_LOGSUMEXP).  Inside a phase each 16-row block
// bi is taken through all of the phase's element-wise ops at once, so only
// its 32 values are live in VGPRs while the rest of the tile stays in the
// accumulator registers.

struct EpiCtx {
  int lane, wm, wn;
  int64_t m0, n0;
  unsigned char* smem;
};

__device__ __forceinline__ int col_local(const EpiCtx& c, int bj) { return c.wn * 128 + bj * 16 + (c.lane >> 4) * 4; }
__device__ __forceinline__ int row_local(const EpiCtx& c, int bi) { return c.wm * 128 + bi * 16 + (c.lane & 15); }

__device__ __forceinline__ bool is_reduction(int kind) {
  return kind == KF_OP_GROUPNORM || kind == KF_OP_ROW_SOFTMAX || kind == KF_OP_ROW_LOGSUMEXP;
}

// 4 consecutive fp32 of a per-column vector (bias, gamma, beta) for block
// bj; columns >= N read 0.
__device__ __forceinline__ f32x4 load_col4(const EpiCtx& c, const float* v, int64_t N, int bj) {
  const __amdgpu_buffer_rsrc_t r = make_rsrc(v + c.n0, (uint32_t)((N - c.n0) * 4));
  return __builtin_bit_cast(f32x4, buf_load16(r, (uint32_t)col_local(c, bj) * 4u));
}

// Reduce one value per 16-row block across the 4 lanes holding each row
// and then across the two waves that share the rows (through LDS).
// `red` holds 2 x 256 floats.  Every thread of the workgroup must call it.
template <bool IS_MAX>
__device__ __forceinline__ void tile_row_reduce(const EpiCtx& c, float (&v)[8], float* red) {
#pragma unroll
  for (int bi = 0; bi < 8; ++bi) {
    float x = v[bi];
    float y = shfl_xor(x, 16);
    x = IS_MAX ? fmaxf(x, y) : x + y;
    y = shfl_xor(x, 32);
    v[bi] = IS_MAX ? fmaxf(x, y) : x + y;
  }
  if (c.lane < 16) {
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) red[c.wn * 256 + row_local(c, bi)] = v[bi];
  }
  __syncthreads();
#pragma unroll
  for (int bi = 0; bi < 8; ++bi) {
    const float o = red[(c.wn ^ 1) * 256 + row_local(c, bi)];
    v[bi] = IS_MAX ? fmaxf(v[bi], o) : v[bi] + o;
  }
  __syncthreads();
}

// Same, but the second (cross-wave) step is skipped: a group of 128 columns
// is exactly one wave's half of the tile row.
__device__ __forceinline__ void wave_row_sum(float (&v)[8]) {
#pragma unroll
  for (int bi = 0; bi < 8; ++bi) {
    float x = v[bi];
    x += shfl_xor(x, 16);
    x += shfl_xor(x, 32);
    v[bi] = x;
  }
}

// Element-wise / tensor-reading ops oi..oe-1 on one 16-row block.
__device__ __forceinline__ void apply_phase(const GemmArgs& p, const EpiCtx& c, int bi, int oi, int oe,
                                            f32x4 (&v)[8]) {
  const int64_t N = p.N;
  for (int o = oi; o < oe; ++o) {
    const EpiOp op = p.prog.op[o];
    switch (op.kind) {
      case KF_OP_BIAS:
#pragma unroll
        for (int bj = 0; bj < 8; ++bj) v[bj] += load_col4(c, p.bias, N, bj);
        break;
      case KF_OP_RESIDUAL_ADD: {
        const int64_t rows = min<int64_t>(BM, p.M - c.m0);
        const int64_t rl = row_local(c, bi);
        if (p.residual_bf16) {
          const uint16_t* base = reinterpret_cast<const uint16_t*>(p.residual) + c.m0 * p.ldr + c.n0;
          const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldr + (N - c.n0)) * 2));
#pragma unroll
          for (int bj = 0; bj < 8; ++bj) {
            const int cl = col_local(c, bj);
            const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldr + cl) * 2) : kOOB;
            const u32x2 w = buf_load8(r, off);
            v[bj] += f32x4{bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
          }
        } else {
          const float* base = reinterpret_cast<const float*>(p.residual) + c.m0 * p.ldr + c.n0;
          const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldr + (N - c.n0)) * 4));
#pragma unroll
          for (int bj = 0; bj < 8; ++bj) {
            const int cl = col_local(c, bj);
            const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldr + cl) * 4) : kOOB;
            v[bj] += __builtin_bit_cast(f32x4, buf_load16(r, off));
          }
        }
        break;
      }
#define KF_EW_CASE(K, EXPR)                          \
  case K:                                            \
    _Pragma("unroll") for (int bj = 0; bj < 8; ++bj) \
    _Pragma("unroll") for (int r = 0; r < 4; ++r) {  \
      const float x = v[bj][r];                      \
      v[bj][r] = (EXPR);                             \
    }                                                \
    break;
      KF_EW_CASE(KF_OP_RELU, fmaxf(x, 0.0f))
      KF_EW_CASE(KF_OP_GELU_TANH, f_gelu_tanh(x))
      KF_EW_CASE(KF_OP_GELU_ERF, f_gelu_erf(x))
      KF_EW_CASE(KF_OP_SWISH, f_swish(x))
      KF_EW_CASE(KF_OP_SIGMOID, f_sigmoid(x))
      KF_EW_CASE(KF_OP_TANH, f_tanh(x))
      KF_EW_CASE(KF_OP_HARDTANH, fminf(fmaxf(x, op.p0), op.p1))
      KF_EW_CASE(KF_OP_SCALE, x * op.p0)
#undef KF_EW_CASE
      default:
        break;
    }
  }
}

__device__ __forceinline__ float sum4(f32x4 a) { return (a[0] + a[1]) + (a[2] + a[3]); }
__device__ __forceinline__ float max4(f32x4 a) { return fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3])); }

// Store one 16-row block (8 x 4 values per lane) to the output tile.
__device__ __forceinline__ void store_block(const GemmArgs& p, const EpiCtx& c, int bi, const f32x4 (&v)[8]) {
  const int64_t N = p.N;
  const int64_t rows = min<int64_t>(BM, p.M - c.m0);
  const int64_t rl = row_local(c, bi);
  if (p.out_bf16) {
    uint16_t* base = reinterpret_cast<uint16_t*>(p.out) + c.m0 * p.ldo + c.n0;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldo + (N - c.n0)) * 2));
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) {
      const int cl = col_local(c, bj);
      const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldo + cl) * 2) : kOOB;
      u32x2 w = {pack_bf16x2(v[bj][0], v[bj][1]), pack_bf16x2(v[bj][2], v[bj][3])};
      buf_store8(w, r, off);
    }
  } else {
    float* base = reinterpret_cast<float*>(p.out) + c.m0 * p.ldo + c.n0;
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base, (uint32_t)(((rows - 1) * p.ldo + (N - c.n0)) * 4));
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) {
      const int cl = col_local(c, bj);
      const uint32_t off = (c.n0 + cl < N) ? (uint32_t)((rl * p.ldo + cl) * 4) : kOOB;
      buf_store16(__builtin_bit_cast(u32x4, v[bj]), r, off);
    }
  }
}

// Epilogue of shape EPI (see EpiShape): ops [0, r) element-wise, op r the
// reduction (if any), ops (r, n) element-wise, then the store.
template <int EPI>
__device__ __forceinline__ void run_epilogue(const GemmArgs& p, const EpiCtx& c, Acc& acc) {
  const int64_t N = p.N;
  float* red = reinterpret_cast<float*>(c.smem);
  const int nops = p.prog.n;
  const int r = EPI == kEpiPlain ? nops : p.red_index;

  if (EPI == kEpiPlain) {
    static_for<0, 8>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      f32x4 v[8];
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) v[bj] = acc[bi][bj] * p.scale;
      apply_phase(p, c, bi, 0, nops, v);
      store_block(p, c, bi, v);
    });
    return;
  }

  // phase A: ops before the reduction, and each row's local statistic
  float st[8];
  static_for<0, 8>([&](auto bi_c) {
    constexpr int bi = decltype(bi_c)::value;
    f32x4 v[8];
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) v[bj] = acc[bi][bj] * p.scale;
    apply_phase(p, c, bi, 0, r, v);
    float s;
    if (EPI == kEpiGroupNorm) {
      s = 0.0f;
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) s += sum4(v[bj]);
    } else {
      // columns past N take no part in a row reduction
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) {
        const int64_t n = c.n0 + col_local(c, bj);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[bj][q] = (n + q < N) ? v[bj][q] : -INFINITY;
      }
      s = -INFINITY;
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) s = fmaxf(s, max4(v[bj]));
    }
    st[bi] = s;
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) acc[bi][bj] = v[bj];
  });

  const EpiOp op = p.prog.op[r];
  if (EPI == kEpiGroupNorm) {
    // group width p.gn_group is 128 (one wave's half of the tile row) or 256
    const bool whole = p.gn_group == 256;
    const float inv_n = 1.0f / (float)p.gn_group;
    if (whole) tile_row_reduce<false>(c, st, red); else wave_row_sum(st);
    float mean[8], ss[8];
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) {
      mean[bi] = st[bi] * inv_n;
      float s = 0.0f;
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) {
        const f32x4 d = acc[bi][bj] - mean[bi];
        s += sum4(d * d);
      }
      ss[bi] = s;
    }
    if (whole) tile_row_reduce<false>(c, ss, red); else wave_row_sum(ss);
    static_for<0, 8>([&](auto bi_c) {
      constexpr int bi = decltype(bi_c)::value;
      const float rs = rsqrtf(ss[bi] * inv_n + op.p0);
      f32x4 v[8];
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) {
        const f32x4 g = load_col4(c, p.gamma, N, bj);
        const f32x4 be = load_col4(c, p.beta, N, bj);
        v[bj] = (acc[bi][bj] - mean[bi]) * rs * g + be;
      }
      apply_phase(p, c, bi, r + 1, nops, v);
      store_block(p, c, bi, v);
    });
    return;
  }

  // kEpiRow: tile-row max, then the sum of e^(h - max); the (max, sum) pair of
  // this 256-column tile goes to the partials buffer.
  tile_row_reduce<true>(c, st, red);
  const bool softmax = op.kind == KF_OP_ROW_SOFTMAX;
  float se[8];
  static_for<0, 8>([&](auto bi_c) {
    constexpr int bi = decltype(bi_c)::value;
    const float ml = st[bi] * kLog2e;
    float s = 0.0f;
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) {
      f32x4 e;
#pragma unroll
      for (int q = 0; q < 4; ++q) e[q] = __builtin_amdgcn_exp2f(fmaf(acc[bi][bj][q], kLog2e, -ml));
      s += sum4(e);
    }
    se[bi] = s;
  });
  tile_row_reduce<false>(c, se, red);
  if (c.lane < 16 && c.wn == 0) {
    float2* part = reinterpret_cast<float2*>(p.partials);
    const int tn = (int)(c.n0 / BN);
#pragma unroll
    for (int bi = 0; bi < 8; ++bi) {
      const int64_t m = c.m0 + row_local(c, bi);
      if (m < p.M) part[m * p.tiles_n + tn] = make_float2(st[bi], se[bi]);
    }
  }
  if (!softmax) return;  // logsumexp: the finishing kernel writes the output
  // softmax: store e^(h - tile max); the row-finishing kernel rescales it
  static_for<0, 8>([&](auto bi_c) {
    constexpr int bi = decltype(bi_c)::value;
    const float ml = st[bi] * kLog2e;
    f32x4 v[8];
#pragma unroll
    for (int bj = 0; bj < 8; ++bj)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[bj][q] = __builtin_amdgcn_exp2f(fmaf(acc[bi][bj][q], kLog2e, -ml));
    store_block(p, c, bi, v);
  });
}

}  // namespace

template <bool B_NK, int EPI>
__global__ __launch_bounds__(NT, 1) void kf_gemm_bf16_256x256(GemmArgs p) {
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1;
  const int wn = wave >> 1;

  int tm, tn;
  tile_coords(blockIdx.x, p.tiles_m, p.tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM;
  const int64_t n0 = (int64_t)tn * BN;
  const int K = (int)p.K;

  // ---- operand descriptors (base at the tile; records end at the last
  // valid element, so rows past M / N read 0)
  const uint16_t* A = reinterpret_cast<const uint16_t*>(p.a);
  const uint16_t* B = reinterpret_cast<const uint16_t*>(p.b);
  const int64_t rows_a = min<int64_t>(BM, p.M - m0);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + m0 * p.lda, (uint32_t)(((rows_a - 1) * p.lda + K) * 2));
  __amdgpu_buffer_rsrc_t rb;
  if (B_NK) {
    const int64_t rows_b = min<int64_t>(BN, p.N - n0);
    rb = make_rsrc(B + n0 * p.ldb, (uint32_t)(((rows_b - 1) * p.ldb + K) * 2));
  } else {
    rb = make_rsrc(B + n0, (uint32_t)((((int64_t)K - 1) * p.ldb + (p.N - n0)) * 2));
  }

  // thread -> staging coordinates
  const int a_row = tid >> 3;   // + 32 i
  const int a_kc = tid & 7;     // 16-byte chunk within the 64-k row
  const int b_kb = tid & 7;     // KN: 8-row k block
  const int b_nb = tid >> 3;    // KN: 8-column n block (0..31)
  const bool b_ncol_ok = B_NK ? true : (n0 + b_nb * 8 < p.N);

  u32x4 sa[8], sb[8];

  auto load_step = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int gk = k0 + a_kc * 8;
      const uint32_t off = gk < K ? (uint32_t)(((int64_t)(a_row + 32 * i) * p.lda + gk) * 2) : kOOB;
      sa[i] = buf_load16(ra, off);
    }
    if (B_NK) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int gk = k0 + a_kc * 8;
        const uint32_t off = gk < K ? (uint32_t)(((int64_t)(a_row + 32 * i) * p.ldb + gk) * 2) : kOOB;
        sb[i] = buf_load16(rb, off);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int gk = k0 + b_kb * 8 + i;
        const uint32_t off = (gk < K && b_ncol_ok) ? (uint32_t)(((int64_t)gk * p.ldb + b_nb * 8) * 2) : kOOB;
        sb[i] = buf_load16(rb, off);
      }
    }
  };

  auto store_step = [&](int stage) {
    unsigned char* sA = smem + stage * kStageBytes;
    unsigned char* sB = sA + kOffB;
#pragma unroll
    for (int i = 0; i < 8; ++i) lds_store(sA + swz(a_row + 32 * i, a_kc), sa[i]);
    if (B_NK) {
#pragma unroll
      for (int i = 0; i < 8; ++i) lds_store(sB + swz(a_row + 32 * i, a_kc), sb[i]);
    } else {
      // 8x8 transpose of bf16: sb[i] holds k = kb*8+i, n = nb*8 .. nb*8+7.
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
        u32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = perm(sb[2 * e + 1][j >> 1], sb[2 * e][j >> 1], sel);
        lds_store(sB + swz(b_nb * 8 + j, b_kb), o);
      }
    }
  };

  Acc acc;
#pragma unroll
  for (int bi = 0; bi < 8; ++bi)
#pragma unroll
    for (int bj = 0; bj < 8; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (K + BK - 1) / BK;
  load_step(0);
  store_step(0);
  __syncthreads();

  for (int t = 0; t < nk; ++t) {
    const int stage = t & 1;
    if (t + 1 < nk) load_step((t + 1) * BK);
    const unsigned char* sA = smem + stage * kStageBytes;
    const unsigned char* sB = sA + kOffB;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int chunk = kk * 4 + (lane >> 4);
      bf16x8 fa[8], fb[8];
#pragma unroll
      for (int bi = 0; bi < 8; ++bi) fa[bi] = lds_load<bf16x8>(sA + swz(wm * 128 + bi * 16 + (lane & 15), chunk));
#pragma unroll
      for (int bj = 0; bj < 8; ++bj) fb[bj] = lds_load<bf16x8>(sB + swz(wn * 128 + bj * 16 + (lane & 15), chunk));
#pragma unroll
      for (int bi = 0; bi < 8; ++bi)
#pragma unroll
        for (int bj = 0; bj < 8; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[bj], fa[bi], acc[bi][bj], 0, 0, 0);
    }
    if (t + 1 < nk) store_step(stage ^ 1);
    __syncthreads();
  }

  EpiCtx c{lane, wm, wn, m0, n0, smem};
  run_epilogue<EPI>(p, c, acc);
}

// ------------------------------------------------------------ host launch

template <bool B_NK>
static void launch_shape(const GemmArgs& p, int epi, dim3 grid, dim3 block, hipStream_t stream) {
  switch (epi) {
    case kEpiGroupNorm:
      hipLaunchKernelGGL((kf_gemm_bf16_256x256<B_NK, kEpiGroupNorm>), grid, block, 0, stream, p);
      break;
    case kEpiRow:
      hipLaunchKernelGGL((kf_gemm_bf16_256x256<B_NK, kEpiRow>), grid, block, 0, stream, p);
      break;
    default:
      hipLaunchKernelGGL((kf_gemm_bf16_256x256<B_NK, kEpiPlain>), grid, block, 0, stream, p);
      break;
  }
}

hipError_t launch_gemm_bf16(const GemmArgs& args, int epi, hipStream_t stream, bool b_nk) {
  GemmArgs p = args;
  p.tiles_m = (int)((p.M + BM - 1) / BM);
  p.tiles_n = (int)((p.N + BN - 1) / BN);
  const dim3 grid(p.tiles_m * p.tiles_n), block(NT);
  if (b_nk)
    launch_shape<true>(p, epi, grid, block, stream);
  else
    launch_shape<false>(p, epi, grid, block, stream);
  return hipGetLastError();
}

int gemm_bf16_tile_n() { return BN; }
int gemm_bf16_tile_m() { return BM; }

}  // namespace kf
