// Device-side building blocks shared by the kf kernels (gfx950 only).
//
// - raw buffer resources: 128-bit loads/stores whose out-of-range lanes read
//   zero / are dropped by the hardware, which is how every kernel handles
//   ragged M, N and K tails without branches;
// - the epilogue op vocabulary and its fp32 math, written from the
//   definitions on the hardware exp2 / rcp instructions;
// - bf16 packing with round-to-nearest-even.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kf_internal.hpp"

namespace kf {

typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(8))) uint32_t u32x8;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) int i32x8;

// ---------------------------------------------------------------- buffers

// Word 3 of a gfx9 buffer descriptor for raw (untyped, stride 0) access.
constexpr int kBufferWord3 = 0x00020000;
// Any voffset at or above this is outside every descriptor we build
// (num_records is always < 2^31), so the access reads 0 / is dropped.
constexpr uint32_t kOOB = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferWord3);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ u32x2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ void buf_store16(u32x4 v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
}
__device__ __forceinline__ void buf_store8(u32x2 v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, 0);
}
__device__ __forceinline__ void buf_store4(uint32_t v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
}

// Streaming (nontemporal) store: the written lines are not kept in the
// caches -- for the outputs of the memory-bound kernels, which no later
// kernel of the same op reads back.  On this GPU a 256 MiB read-and-write
// stream of 16-byte lanes moved at ~4.7 TB/s with ordinary stores and
// ~6.5 TB/s with nontemporal ones: ordinary writes fill the 256 MB
// memory-side cache and evict the lines still to be read.  (The GEMM
// epilogue's 8-byte stores were much slower with the bit, so the matrix-core
// kernels store normally.)
template <typename T>
__device__ __forceinline__ void store_nt(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}

// ------------------------------------------------------------------- bf16

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even: gfx950's v_cvt_pk_bf16_f32
// (the conversion honours the default round-to-nearest-even mode).
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) { return pack_bf16x2(f, 0.0f) & 0xffffu; }

// --------------------------------------------------------------- epilogue math
//
// exp(x) = 2^(x log2 e) on v_exp_f32; 1/x on v_rcp_f32.  Each composite below
// is an identity of the function it computes, arranged so that no
// intermediate overflows to a NaN (large |x| gives +inf in a denominator,
// whose reciprocal is 0).

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float frcp(float x) { return __builtin_amdgcn_rcpf(x); }

// sigmoid(x) = 1 / (1 + e^-x)
__device__ __forceinline__ float f_sigmoid(float x) { return frcp(1.0f + fexp(-x)); }
// swish(x) = x * sigmoid(x)
__device__ __forceinline__ float f_swish(float x) { return x * f_sigmoid(x); }
// tanh(x) = 1 - 2 / (1 + e^(2x))  (e^(2x) = 2^(2 log2 e x); +inf gives 1)
__device__ __forceinline__ float f_tanh(float x) {
  return fmaf(-2.0f, frcp(1.0f + __builtin_amdgcn_exp2f(x * (2.0f * kLog2e))), 1.0f);
}
// 0.5 x (1 + tanh(u)) = x sigmoid(2u) = x / (1 + 2^t), u = sqrt(2/pi) (x +
// 0.044715 x^3), t = -2 u log2 e = x (a + b x^2) with the constants folded
__device__ __forceinline__ float f_gelu_tanh(float x) {
  constexpr float a = -2.0f * 0.7978845608028654f * kLog2e;  // -2 sqrt(2/pi) log2 e
  constexpr float b = a * 0.044715f;
  const float t = x * fmaf(b, x * x, a);
  return x * frcp(1.0f + __builtin_amdgcn_exp2f(t));
}
// erf for the exact GELU, by the rational approximation of Abramowitz and
// Stegun, Handbook of Mathematical Functions, formula 7.1.26 (|error| <=
// 1.5e-7 in exact arithmetic, ~5.5e-7 evaluated in fp32):
//   erf(|x|) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^(-x^2),
//   t = 1 / (1 + p |x|),
// with erf odd.  One reciprocal, one exp and eight fmas, against a library
// erf that evaluates two polynomial branches and selects.  Inside the GELU
// the absolute error is added to 1, so the GELU is within ~3e-7 (relative
// to max(|gelu|, 1)) of its exact value.
__device__ __forceinline__ float f_erf_gelu(float x) {
  constexpr float p = 0.3275911f, a1 = 0.254829592f, a2 = -0.284496736f, a3 = 1.421413741f, a4 = -1.453152027f,
                  a5 = 1.061405429f;
  const float ax = fabsf(x);
  const float t = frcp(fmaf(p, ax, 1.0f));
  const float poly = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, a5, a4), a3), a2), a1);
  const float e = __builtin_amdgcn_exp2f(-(ax * ax) * kLog2e);
  return copysignf(fmaf(-poly, e, 1.0f), x);
}
// exact GELU: 0.5 x (1 + erf(x / sqrt 2))
__device__ __forceinline__ float f_gelu_erf(float x) { return 0.5f * x * (1.0f + f_erf_gelu(x * 0.7071067811865476f)); }
// exact GELU of an input in [-1, 1] (the output of a tanh), by the Maclaurin
// series of erf: 0.5 x (1 + erf(x / sqrt 2)) = 0.5 x + x^2 sum_n e_n x^(2n),
// e_n = 0.5 sqrt(2/pi) (-1)^n / (n! (2n+1) 2^n), summed through n = 6.  On
// [-1, 1] the first omitted term is below 4.2e-8 and the fp32 evaluation is
// within 1.3e-7 of the exact GELU: closer than the general form above, with
// no exp and no reciprocal.
__device__ __forceinline__ float f_gelu_erf_unit(float x) {
  constexpr float e0 = 0.3989422804014327f, e1 = -0.06649038006690546f, e2 = 0.009973557010035817f,
                  e3 = -0.0011873282154804545f, e4 = 0.00011543468761615529f, e5 = -9.444656259503615e-06f,
                  e6 = 6.659693516316651e-07f;
  const float u = x * x;
  const float s = fmaf(u, fmaf(u, fmaf(u, fmaf(u, fmaf(u, fmaf(u, e6, e5), e4), e3), e2), e1), e0);
  return fmaf(u, s, 0.5f * x);
}

// One element-wise op (kinds that need no tensor and no reduction).
__device__ __forceinline__ float apply_elementwise(int kind, float p0, float p1, float x) {
  switch (kind) {
    case KF_OP_RELU: return fmaxf(x, 0.0f);
    case KF_OP_GELU_TANH: return f_gelu_tanh(x);
    case KF_OP_GELU_ERF: return f_gelu_erf(x);
    case KF_OP_SWISH: return f_swish(x);
    case KF_OP_SIGMOID: return f_sigmoid(x);
    case KF_OP_TANH: return f_tanh(x);
    case KF_OP_HARDTANH: return fminf(fmaxf(x, p0), p1);
    case KF_OP_SCALE: return x * p0;
    default: return x;
  }
}

// Apply one element-wise op to a whole register array: the switch is taken
// once per op (the op kind is uniform across the workgroup) and the loop over
// the registers is fully unrolled inside each case.
template <int N>
__device__ __forceinline__ void apply_elementwise_array(int kind, float p0, float p1, float (&v)[N]) {
  switch (kind) {
    case KF_OP_RELU:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = fmaxf(v[i], 0.0f);
      break;
    case KF_OP_GELU_TANH:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = f_gelu_tanh(v[i]);
      break;
    case KF_OP_GELU_ERF:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = f_gelu_erf(v[i]);
      break;
    case KF_OP_SWISH:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = f_swish(v[i]);
      break;
    case KF_OP_SIGMOID:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = f_sigmoid(v[i]);
      break;
    case KF_OP_TANH:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = f_tanh(v[i]);
      break;
    case KF_OP_HARDTANH:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = fminf(fmaxf(v[i], p0), p1);
      break;
    case KF_OP_SCALE:
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = v[i] * p0;
      break;
    default:
      break;
  }
}

__host__ __device__ __forceinline__ bool is_elementwise(int kind) {
  return kind == KF_OP_RELU || kind == KF_OP_GELU_TANH || kind == KF_OP_GELU_ERF ||
         kind == KF_OP_SWISH || kind == KF_OP_SIGMOID || kind == KF_OP_TANH ||
         kind == KF_OP_HARDTANH || kind == KF_OP_SCALE;
}

// The op program held one op per lane (3 VGPRs), loaded once per kernel.  A
// wave-uniform op index then reads the op's fields with v_readlane, where an
// access through the kernel-argument pointer would cost one scalar-memory
// round trip per field and per use.
struct OpTable {
  int kind;
  float p0, p1;
};
__device__ __forceinline__ OpTable load_op_table(const EpiProgram& prog, int lane) {
  OpTable t{0, 0.0f, 0.0f};
  if (lane < KF_MAX_OPS) {
    t.kind = prog.op[lane].kind;
    t.p0 = prog.op[lane].p0;
    t.p1 = prog.op[lane].p1;
  }
  return t;
}
__device__ __forceinline__ int op_kind(const OpTable& t, int o) { return __builtin_amdgcn_readlane(t.kind, o); }
__device__ __forceinline__ float op_p0(const OpTable& t, int o) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(t.p0), o));
}
__device__ __forceinline__ float op_p1(const OpTable& t, int o) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(t.p1), o));
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E), so
// register arrays indexed by I never fall back to scratch memory.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ------------------------------------------------------ accumulator registers

// One MFMA accumulator register read into a VGPR where it is used.  The "a"
// operand keeps the value in its AGPR until this point; with plain element
// reads of a large accumulator array the register allocator copies the whole
// array into VGPRs where the K loop ends, which can overflow them into
// scratch.
__device__ __forceinline__ float acc_read(float a) {
  float v;
  asm("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(a));
  return v;
}

// ---------------------------------------------------------- cross-lane ops

__device__ __forceinline__ float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }

// Sum (or maximum) over aligned groups of `width` lanes (a power of two,
// 1..64); every lane of a group gets the same bits.  Steps within 16 lanes
// use DPP lane moves (quad permutations [1,0,3,2] and [2,3,0,1], then the
// mirror within 8 and within 16 lanes, which pair the same partial results
// as exchanges with lane ^ 4 and lane ^ 8), lane ^ 16 a swizzle, and the two
// halves of the wave are combined from lanes 0 and 32 by readlane; the sums
// are grouped as in an xor butterfly over 1, 2, ..., width / 2.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
template <bool IS_MAX>
__device__ __forceinline__ float lane_group_reduce(float x, int width) {
  auto op = [](float a, float b) { return IS_MAX ? fmaxf(a, b) : a + b; };
  if (width >= 2) x = op(x, dpp_mov<0xB1>(x));   // quad_perm [1,0,3,2]
  if (width >= 4) x = op(x, dpp_mov<0x4E>(x));   // quad_perm [2,3,0,1]
  if (width >= 8) x = op(x, dpp_mov<0x141>(x));  // row_half_mirror
  if (width >= 16) x = op(x, dpp_mov<0x140>(x)); // row_mirror
  if (width >= 32)                               // lane ^ 16 within 32 lanes
    x = op(x, __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x), 0x1F | (0x10 << 10))));
  if (width >= 64) {
    const float lo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
    const float hi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
    x = op(lo, hi);
  }
  return x;
}

}  // namespace kf
