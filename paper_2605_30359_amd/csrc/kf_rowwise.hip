// Row-wise op chains with no contraction (h = A): the memory-bound reduction
// operators of the paper's category table (Table 2: reduction-dominated
// chains -- softmax, logsumexp, GroupNorm with their element-wise
// neighbours), following its advice for them (Appendix B: hierarchical
// reductions, normalise before exponentiating).  The whole row stays in
// registers between the passes, so A (and a residual) is read once and the
// output written once: the kernel's roofline is HBM bandwidth.
//
//   layout   one workgroup of 256 threads per row; the row is taken as
//            16-byte chunks of 8 values, chunk c held by thread c % 256 in
//            register slot c / 256, so every load and store instruction of a
//            wave covers contiguous memory
//   row max / sum   per thread over its chunks, then across the wave (xor
//            exchanges), then the four waves through LDS, in a fixed order
//   GroupNorm   per-chunk sums, combined per group in a fixed order: as a
//            row reduction (one group per row), by xor exchanges among the
//            lanes of a group (up to 64 chunks, a power of two), or by a
//            pairwise tree in LDS (any group width that is a multiple of 8
//            columns); the mean and the biased variance take two such passes
//            over the registers
#include <algorithm>

#include "kf_device.hpp"
#include "kf_launch.hpp"

namespace kf {

namespace {

constexpr int RT = 256;                   // threads per workgroup (one row)
constexpr int kMaxCols = 16384;
constexpr int kMaxChunks = kMaxCols / 8;  // 2048 chunks of 8 values
constexpr int kSlots = kMaxChunks / RT;   // at most 8 chunks per thread

typedef float Chunk[8];

// Row-wide max or sum of one value per thread; every thread gets the result.
template <bool IS_MAX>
__device__ __forceinline__ float row_reduce(float v, float* red) {
  v = lane_group_reduce<IS_MAX>(v, 64);
  __syncthreads();  // the previous reduction's readers are done with red
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < RT / 64; ++w) r = IS_MAX ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

// NT: a streaming (nontemporal) load, for data read once
template <bool NT = false>
__device__ __forceinline__ void load_chunk(const void* base, bool bf16, int64_t off, Chunk& x) {
  if (bf16) {
    const u32x4* q = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(base) + off);
    const u32x4 w = NT ? __builtin_nontemporal_load(q) : *q;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = bf16_lo(w[e]);
      x[2 * e + 1] = bf16_hi(w[e]);
    }
  } else {
    const f32x4* f = reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(base) + off);
    const f32x4 lo = f[0], hi = f[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = lo[e];
      x[4 + e] = hi[e];
    }
  }
}

}  // namespace

// S = register slots per thread (chunks of the row / 256, rounded up); CH a
// compile-time op chain (0: the op list is interpreted)
template <int S, int CH>
__global__ __launch_bounds__(RT) void kf_rowwise(RowArgs p) {
  __shared__ float part[kMaxChunks];  // per-chunk partial sums (GroupNorm)
  __shared__ float red[RT / 64];
  const int t = threadIdx.x;
  const int64_t m = blockIdx.x;
  const int chunks = (int)(p.N >> 3);
  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, t & 63);

  Chunk v[S];
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int c = j * RT + t;
    if (c < chunks) load_chunk(p.a, p.in_bf16 != 0, m * p.lda + c * 8, v[j]);
  }

  // op o of kind `kind`; true once a row logsumexp has written the result
  auto run_op = [&](int kind, int o) -> bool {
    if (kind == KF_OP_BIAS) {
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
        const f32x4* b = reinterpret_cast<const f32x4*>(p.bias + c * 8);
        const f32x4 lo = b[0], hi = b[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[j][e] += lo[e];
          v[j][4 + e] += hi[e];
        }
      }
    } else if (kind == KF_OP_RESIDUAL_ADD) {
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
        Chunk r;
        load_chunk(p.residual, p.residual_bf16 != 0, m * p.ldr + c * 8, r);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] += r[e];
      }
    } else if (kind == KF_OP_GROUPNORM) {
      const int L = p.gn_group >> 3;  // chunks per group
      const float inv_n = 1.0f / (float)p.gn_group;
      const float eps = op_p0(ops, o);
      // Replace the per-chunk values q[j] by the sums over their groups.
      // One group per row: a row reduction.  A power-of-two number of chunks
      // up to 64: the group is L consecutive lanes of one wave (256 % L == 0
      // aligns it), summed by xor exchanges -- each level adds two operands
      // in both of their lanes, so every lane ends with the same bits.
      // Otherwise a pairwise tree over the chunks in LDS.
      auto group_sums = [&](float (&q)[S]) {
        if (L == chunks) {
          float s = 0.0f;
#pragma unroll
          for (int j = 0; j < S; ++j) s += q[j];
          s = row_reduce<false>(s, red);
#pragma unroll
          for (int j = 0; j < S; ++j) q[j] = s;
        } else if ((L & (L - 1)) == 0 && L <= 64) {
#pragma unroll
          for (int j = 0; j < S; ++j) q[j] = lane_group_reduce<false>(q[j], L);
        } else {
#pragma unroll
          for (int j = 0; j < S; ++j) {
            const int c = j * RT + t;
            if (c < chunks) part[c] = q[j];
          }
          for (int s = 1; s < L; s <<= 1) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < S; ++j) {
              const int c = j * RT + t;
              const int cg = c % L;
              if (c < chunks && (cg & (2 * s - 1)) == 0 && cg + s < L) part[c] += part[c + s];
            }
          }
          __syncthreads();
#pragma unroll
          for (int j = 0; j < S; ++j) {
            const int c = j * RT + t;
            q[j] = c < chunks ? part[c - c % L] : 0.0f;
          }
          __syncthreads();  // every thread has read part[] before it is reused
        }
      };
      float mean[S], rs[S];
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        mean[j] = c < chunks ? ((v[j][0] + v[j][1]) + (v[j][2] + v[j][3])) + ((v[j][4] + v[j][5]) + (v[j][6] + v[j][7]))
                             : 0.0f;
      }
      group_sums(mean);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        mean[j] *= inv_n;
        float q = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = v[j][e] - mean[j];
          q = fmaf(d, d, q);
        }
        rs[j] = c < chunks ? q : 0.0f;
      }
      group_sums(rs);
#pragma unroll
      for (int j = 0; j < S; ++j) rs[j] = rsqrtf(rs[j] * inv_n + eps);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
        const f32x4* g = reinterpret_cast<const f32x4*>(p.gamma + c * 8);
        const f32x4* b = reinterpret_cast<const f32x4*>(p.beta + c * 8);
        const f32x4 g0 = g[0], g1 = g[1], b0 = b[0], b1 = b[1];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[j][e] = fmaf((v[j][e] - mean[j]) * rs[j], g0[e], b0[e]);
          v[j][4 + e] = fmaf((v[j][4 + e] - mean[j]) * rs[j], g1[e], b1[e]);
        }
      }
    } else if (is_row_op(kind)) {
      // the last op: max, then the sum of e^(h - max)
      // cross-entropy: the thread holding column t (chunk t / 8, slot
      // chunk / 256) keeps h[t] before the exponentials replace it
      int32_t tgt = -1;
      float ht = 0.0f;
      if (kind == KF_OP_ROW_CROSS_ENTROPY) {
        tgt = p.targets[m];
#pragma unroll
        for (int j = 0; j < S; ++j) {
          const int c = j * RT + t;
#pragma unroll
          for (int e = 0; e < 8; ++e) ht = (tgt >= 0 && tgt < p.N && tgt == c * 8 + e) ? v[j][e] : ht;
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, v[j][e]);
      }
      mx = row_reduce<true>(mx, red);
      const float ml = mx * kLog2e;
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[j][e] = __builtin_amdgcn_exp2f(fmaf(v[j][e], kLog2e, -ml));
          s += v[j][e];
        }
      }
      s = row_reduce<false>(s, red);
      if (kind == KF_OP_ROW_LOGSUMEXP) {
        if (t == 0) reinterpret_cast<float*>(p.out)[m] = mx + logf(s);
        return true;
      }
      if (kind == KF_OP_ROW_CROSS_ENTROPY) {
        const bool valid = tgt >= 0 && tgt < p.N;
        if (valid ? ((tgt >> 3) % RT == t) : t == 0)
          reinterpret_cast<float*>(p.out)[m] = valid ? (mx + logf(s)) - ht : __builtin_nanf("");
        return true;
      }
      const float inv = 1.0f / s;
#pragma unroll
      for (int j = 0; j < S; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] *= inv;
    } else {
      const float p0 = op_p0(ops, o), p1 = op_p1(ops, o);
#pragma unroll
      for (int j = 0; j < S; ++j) {
        const int c = j * RT + t;
        if (c >= chunks) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) v[j][e] = apply_elementwise(kind, p0, p1, v[j][e]);
      }
    }
    return false;
  };
  if constexpr (CH == 0) {
    for (int o = 0; o < nops; ++o)
      if (run_op(op_kind(ops, o), o)) return;
  } else {
    bool done = false;
    static_for<0, kChainLen[CH]>([&](auto O_c) {
      constexpr int o = decltype(O_c)::value;
      if (!done) done = run_op(kChainOps[CH][o], o);
    });
    if (done) return;
  }

#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int c = j * RT + t;
    if (c >= chunks) continue;
    if (p.out_bf16) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(v[j][2 * e], v[j][2 * e + 1]);
      store_nt(reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(p.out) + m * p.ldo + c * 8), w);
    } else {
      f32x4* f = reinterpret_cast<f32x4*>(reinterpret_cast<float*>(p.out) + m * p.ldo + c * 8);
      store_nt(f, f32x4{v[j][0], v[j][1], v[j][2], v[j][3]});
      store_nt(f + 1, f32x4{v[j][4], v[j][5], v[j][6], v[j][7]});
    }
  }
}


// GroupNorm chains whose group is a power-of-two number of chunks up to 64
// (group widths 8..512 columns), with element-wise ops, a bias and a
// residual add around the GroupNorm but no whole-row reduction.  The groups
// are independent, so the work is cut into column panels instead of rows:
// a wave owns one 512-column panel of P = 64 / L groups (lane = group-in-
// panel * L + chunk-in-group) for its whole life and walks rows, one row per
// step, and the four waves of a workgroup own four adjacent panels, so each
// step of a workgroup reads 2048 contiguous columns of a row.  gamma and
// beta (and the bias) of a lane's 8 columns are loaded once into registers
// -- a row kernel re-reads them for every row, 64 KiB per row at 8192
// columns -- and the group statistics are sums over L lanes by xor
// exchanges (no LDS, no barrier).  One row per step: the kernel needs few
// registers, so a CU holds eight waves per SIMD, and more waves with a row
// each kept more bytes in flight than fewer waves with several rows each
// (four rows per step ran F3 in 74 us, two in 68, one in 64; one row with
// the next one requested ahead, 68).
template <int CH>
__global__ __launch_bounds__(RT) void kf_rowwise_gn_panel(RowArgs p) {
  const int lane = threadIdx.x & 63;
  const int L = p.gn_group >> 3;  // chunks per group: a power of two, 1..64
  const int P = 64 / L;           // groups per panel
  const int groups = (int)(p.N / p.gn_group);
  const int panels = (groups + P - 1) / P;
  const int panel_sets = (panels + RT / 64 - 1) / (RT / 64);
  const int panel = (int)(blockIdx.x % panel_sets) * (RT / 64) + (threadIdx.x >> 6);
  if (panel >= panels) return;  // no barrier below
  const int64_t row_stride = gridDim.x / panel_sets;
  const int64_t row0 = blockIdx.x / panel_sets;
  const int q = lane & (L - 1);
  const int grp = panel * P + lane / L;
  const bool live = grp < groups;
  const int64_t col = (int64_t)(live ? grp : 0) * p.gn_group + q * 8;
  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const float inv_n = 1.0f / (float)p.gn_group;

  float gam[8], bet[8], bia[8];
  {
    const f32x4* gp = reinterpret_cast<const f32x4*>(p.gamma + col);
    const f32x4* bp = reinterpret_cast<const f32x4*>(p.beta + col);
    const f32x4 g0 = gp[0], g1 = gp[1], b0 = bp[0], b1 = bp[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      gam[e] = g0[e];
      gam[4 + e] = g1[e];
      bet[e] = b0[e];
      bet[4 + e] = b1[e];
      bia[e] = bia[4 + e] = 0.0f;
    }
    if (p.bias) {
      const f32x4* cp = reinterpret_cast<const f32x4*>(p.bias + col);
      const f32x4 c0 = cp[0], c1 = cp[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bia[e] = c0[e];
        bia[4 + e] = c1[e];
      }
    }
  }

  // sum over the L lanes of this lane's group (every lane gets the same bits)
  auto group_sum = [&](float x) { return lane_group_reduce<false>(x, L); };

  auto compute_store = [&](int64_t row, Chunk& v, const Chunk& r) {
    auto run_op = [&](int kind, int o) {
      if (kind == KF_OP_BIAS) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += bia[e];
      } else if (kind == KF_OP_RESIDUAL_ADD) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += r[e];
      } else if (kind == KF_OP_GROUPNORM) {
        const float eps = op_p0(ops, o);
        const float sum = ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
        const float mean = group_sum(sum) * inv_n;
        float qd = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = v[e] - mean;
          qd = fmaf(d, d, qd);
        }
        const float rs = rsqrtf(group_sum(qd) * inv_n + eps);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = fmaf((v[e] - mean) * rs, gam[e], bet[e]);
      } else {
        apply_elementwise_array<8>(kind, op_p0(ops, o), op_p1(ops, o), v);
      }
    };
    if constexpr (CH == 0) {
      for (int o = 0; o < nops; ++o) run_op(op_kind(ops, o), o);
    } else {
      static_for<0, kChainLen[CH]>([&](auto O_c) {
        constexpr int o = decltype(O_c)::value;
        run_op(kChainOps[CH][o], o);
      });
    }
    if (!live) return;
    if (p.out_bf16) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(v[2 * e], v[2 * e + 1]);
      store_nt(reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(p.out) + row * p.ldo + col), w);
    } else {
      f32x4* f = reinterpret_cast<f32x4*>(reinterpret_cast<float*>(p.out) + row * p.ldo + col);
      store_nt(f, f32x4{v[0], v[1], v[2], v[3]});
      store_nt(f + 1, f32x4{v[4], v[5], v[6], v[7]});
    }
  };

  for (int64_t row = row0; row < p.M; row += row_stride) {
    Chunk v, r;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = r[e] = 0.0f;
    if (live) {
      load_chunk(p.a, p.in_bf16 != 0, row * p.lda + col, v);
      if (p.residual) load_chunk(p.residual, p.residual_bf16 != 0, row * p.ldr + col, r);
    }
    compute_store(row, v, r);
  }
}

// Row logsumexp and cross-entropy (a row op that reduces the row to one
// value, after element-wise ops and a bias): no output row, so the row is
// streamed instead of held.  One wave per row; lane l takes chunks l,
// l + 64, ... in groups of kStreamUnroll (all loads of a group issued
// together), keeping a running (max, sum of e^(h - max)) that is rescaled
// when the maximum grows -- once per group, by the group's maximum.  The
// wave then combines its lanes' pairs; cross-entropy subtracts h[t], which
// the lane holding chunk t / 8 picked up on the way.  Any row length; few
// registers, so eight waves per SIMD each keep a group of loads in flight
// (F5's 8192 x 16384 bf16 rows: groups of 1 or 2 chunks 46.6 us a step,
// 4 chunks 52, 8 chunks 47; streaming loads 46.0).
constexpr int kStreamUnroll = 2;

template <int CH>
__global__ __launch_bounds__(RT) void kf_row_reduce_stream(RowArgs p) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (RT / 64);
  const int nops = p.prog.n;
  const OpTable ops = load_op_table(p.prog, lane);
  const int64_t chunks = p.N >> 3;
  const int last = (CH == 0 ? nops : kChainLen[CH]) - 1;
  const int row_kind = CH == 0 ? op_kind(ops, last) : kChainOps[CH][kChainLen[CH] > 0 ? kChainLen[CH] - 1 : 0];
  const bool ce = row_kind == KF_OP_ROW_CROSS_ENTROPY;

  for (int64_t m = (int64_t)blockIdx.x * (RT / 64) + (threadIdx.x >> 6); m < p.M; m += waves) {
    const int32_t tgt = ce ? p.targets[m] : -1;
    const bool valid = tgt >= 0 && tgt < p.N;
    const int64_t tchunk = valid ? (tgt >> 3) : -1;
    float mx = -INFINITY, sum = 0.0f, ht = 0.0f;
    for (int64_t c0 = lane; c0 < chunks; c0 += 64 * kStreamUnroll) {
      Chunk v[kStreamUnroll];
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u) {
        const int64_t c = c0 + 64 * u;
        if (c < chunks) {
          load_chunk<true>(p.a, p.in_bf16 != 0, m * p.lda + c * 8, v[u]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[u][e] = -INFINITY;
        }
      }
      // the element-wise ops (and the bias) before the row op
      auto run_op = [&](int kind, int o) {
#pragma unroll
        for (int u = 0; u < kStreamUnroll; ++u) {
          const int64_t c = c0 + 64 * u;
          if (c >= chunks) continue;
          if (kind == KF_OP_BIAS) {
            const f32x4* b = reinterpret_cast<const f32x4*>(p.bias + c * 8);
            const f32x4 lo = b[0], hi = b[1];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[u][e] += lo[e];
              v[u][4 + e] += hi[e];
            }
          } else {
            apply_elementwise_array<8>(kind, op_p0(ops, o), op_p1(ops, o), v[u]);
          }
        }
      };
      if constexpr (CH == 0) {
        for (int o = 0; o < last; ++o) run_op(op_kind(ops, o), o);
      } else {
        static_for<0, kChainLen[CH] - 1>([&](auto O_c) {
          constexpr int o = decltype(O_c)::value;
          run_op(kChainOps[CH][o], o);
        });
      }
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u)
        if (c0 + 64 * u == tchunk) {
#pragma unroll
          for (int e = 0; e < 8; ++e) ht = (tgt & 7) == e ? v[u][e] : ht;
        }
      float gm = mx;
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) gm = fmaxf(gm, v[u][e]);
      if (gm == -INFINITY) continue;  // nothing but -inf so far
      const float gl = gm * kLog2e;
      float gs = 0.0f;
#pragma unroll
      for (int u = 0; u < kStreamUnroll; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) gs += __builtin_amdgcn_exp2f(fmaf(v[u][e], kLog2e, -gl));
      sum = (mx == -INFINITY ? 0.0f : sum * __builtin_amdgcn_exp2f(fmaf(mx, kLog2e, -gl))) + gs;
      mx = gm;
    }
    // combine the lanes: the row maximum, then each lane's sum rescaled to it
    const float rmx = lane_group_reduce<true>(mx, 64);
    const float part = mx == -INFINITY ? 0.0f : sum * __builtin_amdgcn_exp2f(fmaf(mx, kLog2e, -rmx * kLog2e));
    const float rsum = lane_group_reduce<false>(part, 64);
    const float lse = rmx + logf(rsum);
    if (ce) {
      const float h = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ht), valid ? (int)(tchunk & 63) : 0));
      if (lane == 0) reinterpret_cast<float*>(p.out)[m] = valid ? lse - h : __builtin_nanf("");
    } else if (lane == 0) {
      reinterpret_cast<float*>(p.out)[m] = lse;
    }
  }
}

namespace {

// The column-panel form applies to a GroupNorm chain with no whole-row op
// whose group is 1, 2, 4, ..., 64 chunks of 8 columns.
bool panel_applies(const RowArgs& a) {
  if (a.gn_group <= 0 || a.gn_group % 8 || a.gn_group > 512) return false;
  const int L = a.gn_group / 8;
  if (L & (L - 1)) return false;
  for (int i = 0; i < a.prog.n; ++i) {
    const int k = a.prog.op[i].kind;
    if (is_row_op(k)) return false;
  }
  return true;
}

template <int CH>
hipError_t launch_panel(const RowArgs& args, hipStream_t stream) {
  // as many workgroups as the device holds at once, whole sets of them per
  // four adjacent panels, and no more workgroups per set than rows
  static const int resident = resident_blocks(kf_rowwise_gn_panel<CH>, RT);
  const int64_t groups = args.N / args.gn_group;
  const int64_t P = 64 / (args.gn_group / 8);
  const int64_t panels = (groups + P - 1) / P;
  const int64_t panel_sets = (panels + RT / 64 - 1) / (RT / 64);
  int64_t per_set = std::max<int64_t>(1, resident / panel_sets);
  per_set = std::min<int64_t>(per_set, args.M);
  const dim3 grid((unsigned)(panel_sets * per_set)), block(RT);
  hipLaunchKernelGGL((kf_rowwise_gn_panel<CH>), grid, block, 0, stream, args);
  return hipGetLastError();
}

template <int CH>
hipError_t launch_stream(const RowArgs& args, hipStream_t stream) {
  static const int resident = resident_blocks(kf_row_reduce_stream<CH>, RT);
  const int64_t need = (args.M + RT / 64 - 1) / (RT / 64);
  const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, resident))), block(RT);
  hipLaunchKernelGGL((kf_row_reduce_stream<CH>), grid, block, 0, stream, args);
  return hipGetLastError();
}

template <int CH>
hipError_t launch_rowwise_chain(const RowArgs& args, hipStream_t stream) {
  const int64_t slots = (args.N / 8 + RT - 1) / RT;
  const dim3 grid((unsigned)args.M), block(RT);
  if (slots <= 1)
    hipLaunchKernelGGL((kf_rowwise<1, CH>), grid, block, 0, stream, args);
  else if (slots <= 2)
    hipLaunchKernelGGL((kf_rowwise<2, CH>), grid, block, 0, stream, args);
  else if (slots <= 4)
    hipLaunchKernelGGL((kf_rowwise<4, CH>), grid, block, 0, stream, args);
  else if (slots <= kSlots)
    hipLaunchKernelGGL((kf_rowwise<kSlots, CH>), grid, block, 0, stream, args);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

// The benchmarked row chains (GroupNorm + swish + residual, softmax) run an
// epilogue generated for exactly that op sequence; any other list runs
// interpreted.
hipError_t launch_rowwise(const RowArgs& args, int chain, hipStream_t stream) {
  if (args.M <= 0) return hipSuccess;
  if (row_reduce_streams(args.prog)) {
    switch (chain) {
      case kChainRowLogsumexp: return launch_stream<kChainRowLogsumexp>(args, stream);
      case kChainRowCrossEntropy: return launch_stream<kChainRowCrossEntropy>(args, stream);
      default: return launch_stream<0>(args, stream);
    }
  }
  if (panel_applies(args)) {
    switch (chain) {
      case 5: return launch_panel<5>(args, stream);
      case kChainGroupNorm: return launch_panel<kChainGroupNorm>(args, stream);
      default: return launch_panel<0>(args, stream);
    }
  }
  switch (chain) {
    case 5: return launch_rowwise_chain<5>(args, stream);
    case kChainRowSoftmax: return launch_rowwise_chain<kChainRowSoftmax>(args, stream);
    case kChainGroupNorm: return launch_rowwise_chain<kChainGroupNorm>(args, stream);
    case kChainRowLogsumexp: return launch_rowwise_chain<kChainRowLogsumexp>(args, stream);
    case kChainRowCrossEntropy: return launch_rowwise_chain<kChainRowCrossEntropy>(args, stream);
    default: return launch_rowwise_chain<0>(args, stream);
  }
}

int rowwise_max_cols() { return kMaxCols; }

const char* rowwise_kernel(const EpiProgram& prog, int gn_group) {
  RowArgs a{};
  a.prog = prog;
  a.gn_group = gn_group;
  return row_reduce_streams(prog) ? "kf_row_reduce_stream" : panel_applies(a) ? "kf_rowwise_gn_panel" : "kf_rowwise";
}

// The streamed form applies to a list that ends with a row logsumexp or
// cross-entropy and has only element-wise ops and a bias before it.
bool row_reduce_streams(const EpiProgram& prog) {
  const int n = prog.n;
  if (n < 1) return false;
  const int k = prog.op[n - 1].kind;
  if (k != KF_OP_ROW_LOGSUMEXP && k != KF_OP_ROW_CROSS_ENTROPY) return false;
  for (int i = 0; i + 1 < n; ++i) {
    const int o = prog.op[i].kind;
    if (o != KF_OP_BIAS && !is_elementwise(o)) return false;
  }
  return true;
}

}  // namespace kf
