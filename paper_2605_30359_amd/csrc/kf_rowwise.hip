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
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float y = shfl_xor(v, o);
    v = IS_MAX ? fmaxf(v, y) : v + y;
  }
  __syncthreads();  // the previous reduction's readers are done with red
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < RT / 64; ++w) r = IS_MAX ? fmaxf(r, red[w]) : r + red[w];
  return r;
}

__device__ __forceinline__ void load_chunk(const void* base, bool bf16, int64_t off, Chunk& x) {
  if (bf16) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(base) + off);
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
          for (int d = 1; d < L; d <<= 1)
#pragma unroll
            for (int j = 0; j < S; ++j) q[j] += shfl_xor(q[j], d);
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
// each wave takes one group g for its whole life and walks rows, P = 64 / L
// rows per step (lane = row-in-step * L + chunk-in-group).  gamma and beta
// (and the bias) of the wave's 8 columns per lane are loaded once into
// registers -- a row kernel re-reads them for every row, 64 KiB per row at
// 8192 columns -- and the group statistics are sums over L lanes by xor
// exchanges (no LDS, no barrier).  Each lane keeps kPanelUnroll steps of A
// (and residual) chunks in flight.
constexpr int kPanelUnroll = 4;

template <int CH>
__global__ __launch_bounds__(RT) void kf_rowwise_gn_panel(RowArgs p) {
  const int lane = threadIdx.x & 63;
  const int L = p.gn_group >> 3;  // chunks per group: a power of two, 1..64
  const int P = 64 / L;           // rows per step
  const int groups = (int)(p.N / p.gn_group);
  const int g = blockIdx.x % groups;
  const int waves = (int)(gridDim.x / groups) * (RT / 64);
  const int wave = (int)(blockIdx.x / groups) * (RT / 64) + (threadIdx.x >> 6);
  const int q = lane & (L - 1);
  const int pr = lane / L;
  const int64_t col = (int64_t)g * p.gn_group + q * 8;
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
  auto group_sum = [&](float x) {
    for (int d = 1; d < L; d <<= 1) x += shfl_xor(x, d);
    return x;
  };

  const int64_t steps = (p.M + P - 1) / P;
  for (int64_t s0 = wave; s0 < steps; s0 += (int64_t)waves * kPanelUnroll) {
    Chunk v[kPanelUnroll], r[kPanelUnroll];
    int64_t row[kPanelUnroll];
    bool ok[kPanelUnroll];
#pragma unroll
    for (int u = 0; u < kPanelUnroll; ++u) {
      row[u] = (s0 + (int64_t)u * waves) * P + pr;
      ok[u] = s0 + (int64_t)u * waves < steps && row[u] < p.M;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[u][e] = r[u][e] = 0.0f;
      if (ok[u]) {
        load_chunk(p.a, p.in_bf16 != 0, row[u] * p.lda + col, v[u]);
        if (p.residual) load_chunk(p.residual, p.residual_bf16 != 0, row[u] * p.ldr + col, r[u]);
      }
    }
    auto run_op = [&](int kind, int o) {
#pragma unroll
      for (int u = 0; u < kPanelUnroll; ++u) {
        if (kind == KF_OP_BIAS) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[u][e] += bia[e];
        } else if (kind == KF_OP_RESIDUAL_ADD) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[u][e] += r[u][e];
        } else if (kind == KF_OP_GROUPNORM) {
          const float eps = op_p0(ops, o);
          const float sum = ((v[u][0] + v[u][1]) + (v[u][2] + v[u][3])) + ((v[u][4] + v[u][5]) + (v[u][6] + v[u][7]));
          const float mean = group_sum(sum) * inv_n;
          float qd = 0.0f;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float d = v[u][e] - mean;
            qd = fmaf(d, d, qd);
          }
          const float rs = rsqrtf(group_sum(qd) * inv_n + eps);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[u][e] = fmaf((v[u][e] - mean) * rs, gam[e], bet[e]);
        } else {
          apply_elementwise_array<8>(kind, op_p0(ops, o), op_p1(ops, o), v[u]);
        }
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
#pragma unroll
    for (int u = 0; u < kPanelUnroll; ++u) {
      if (!ok[u]) continue;
      if (p.out_bf16) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(v[u][2 * e], v[u][2 * e + 1]);
        store_nt(reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(p.out) + row[u] * p.ldo + col), w);
      } else {
        f32x4* f = reinterpret_cast<f32x4*>(reinterpret_cast<float*>(p.out) + row[u] * p.ldo + col);
        store_nt(f, f32x4{v[u][0], v[u][1], v[u][2], v[u][3]});
        store_nt(f + 1, f32x4{v[u][4], v[u][5], v[u][6], v[u][7]});
      }
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
  // column group, and no more waves per group than it has row steps
  static const int resident = resident_blocks(kf_rowwise_gn_panel<CH>, RT);
  const int64_t groups = args.N / args.gn_group;
  const int64_t P = 64 / (args.gn_group / 8);
  const int64_t steps = (args.M + P - 1) / P;
  int64_t per_group = std::max<int64_t>(1, resident / groups);
  per_group = std::min<int64_t>(per_group, (steps + RT / 64 - 1) / (RT / 64));
  const dim3 grid((unsigned)(groups * per_group)), block(RT);
  hipLaunchKernelGGL((kf_rowwise_gn_panel<CH>), grid, block, 0, stream, args);
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

}  // namespace kf
