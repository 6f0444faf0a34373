// Shared device helpers for the gfx950 kernels: storage types, bf16 rounding,
// MFMA wrappers, wave/block reductions and the XCD-aware block remap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

typedef uint16_t bf16_t;   // raw bfloat16 bit pattern

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef double f64x2_t __attribute__((ext_vector_type(2)));
// 16 bytes in four 32-bit lanes; native vector type so values stay in VGPRs.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int WAVE = 64;

// ---------------------------------------------------------------- bf16 ----
// float -> bfloat16 with round to nearest even, two at a time through the
// gfx950 conversion instruction (v_cvt_pk_bf16_f32); NaN stays NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)(pack_bf2(f, 0.f) & 0xffffu); }
__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// ---------------------------------------------------------------- fp16 ----
// IEEE binary16 product operands (a tag type: the bits live in packed words).
// float -> fp16 rounds to nearest even.
struct f16_t {
  uint16_t bits;
};
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ uint32_t pack_h2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, f16x2_t));
}

// ------------------------------------------------- iterate state ----------
// The bf16 iterate is stored as hi = bf16(x) plus one residual byte: the OCP
// float8 e4m3 ("fn") code of (x - hi) 2^16, clamped to +-448 and rounded to
// nearest even, read back as hi + e4m3 2^-16. The gfx950 scaled conversions
// divide by the scale when encoding and multiply by it when decoding, exactly
// for a power of two; the clamp keeps the encoder away from its NaN code.
// x - hi is exact in fp32 (hi is x rounded to 8 significant bits).
constexpr float STATE_SCALE = 0x1p-16f;
constexpr float STATE_LIM = 448.f * 0x1p-16f;
typedef short short2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float state_clamp(float d) { return __builtin_amdgcn_fmed3f(d, -STATE_LIM, STATE_LIM); }
// residuals x_i - hi_i of four consecutive elements -> one word (element i in byte i)
__device__ __forceinline__ uint32_t state_pack4(float d0, float d1, float d2, float d3) {
  short2_t w = {0, 0};
  w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, state_clamp(d0), state_clamp(d1), STATE_SCALE, false);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(w, state_clamp(d2), state_clamp(d3), STATE_SCALE, true);
  return __builtin_bit_cast(uint32_t, w);
}
// residual (x - hi) of the element in byte I of a word
template <int I>
__device__ __forceinline__ float state_res(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_f32_fp8((int)w, STATE_SCALE, I);
}
// eight consecutive elements: values v, their bf16 words nh (two per word)
// -> eight residual bytes
__device__ __forceinline__ u32x2_t state_pack8(const float (&v)[8], const uint32_t (&nh)[4]) {
  float d[8];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    d[2 * q] = v[2 * q] - __uint_as_float(nh[q] << 16);
    d[2 * q + 1] = v[2 * q + 1] - __uint_as_float(nh[q] & 0xffff0000u);
  }
  return u32x2_t{state_pack4(d[0], d[1], d[2], d[3]), state_pack4(d[4], d[5], d[6], d[7])};
}
// hi (two bf16 per word) + residual bytes -> the carried values of eight elements
__device__ __forceinline__ void state_value8(const uint32_t (&h)[4], uint32_t l0, uint32_t l1, float (&x)[8]) {
  const float r[8] = {state_res<0>(l0), state_res<1>(l0), state_res<2>(l0), state_res<3>(l0),
                      state_res<0>(l1), state_res<1>(l1), state_res<2>(l1), state_res<3>(l1)};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    x[2 * q] = __uint_as_float(h[q] << 16) + r[2 * q];
    x[2 * q + 1] = __uint_as_float(h[q] & 0xffff0000u) + r[2 * q + 1];
  }
}

// Component i (a compile-time constant after unrolling) of a 16-byte value.
__device__ __forceinline__ uint32_t u4c(const u32x4_t& u, int i) { return u[i]; }
__device__ __forceinline__ float u4f(const u32x4_t& u, int i) { return __uint_as_float(u[i]); }
__device__ __forceinline__ u32x4_t ld16(const void* p) { return *reinterpret_cast<const u32x4_t*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4_t& v) { *reinterpret_cast<u32x4_t*>(p) = v; }
// Streaming (non-temporal) stores, for large results that are not read again
// soon: they do not hold L2 lines for write-back, which otherwise competes
// with the operand traffic of concurrently running GEMM main loops (measured:
// the iterate update's state stores cost about 13% less time this way).
__device__ __forceinline__ void st16_nt(void* p, const u32x4_t& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t*>(p));
}
__device__ __forceinline__ void st8_nt(void* p, const u32x2_t& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x2_t*>(p));
}
// Streaming when NT, else an ordinary store (for a result the next launch
// reads at once and that fits in the last-level cache). A compile-time
// choice: with a run-time flag the compiler merges the two stores into one
// and the non-temporal hint is lost.
template <bool NT>
__device__ __forceinline__ void st16_pol(void* p, const u32x4_t& v) {
  if constexpr (NT) st16_nt(p, v);
  else st16(p, v);
}

// Element traits: storage type -> float and back.
template <typename T> struct Cvt;
template <> struct Cvt<float> {
  __device__ __forceinline__ static float to_f(float v) { return v; }
  __device__ __forceinline__ static float from_f(float v) { return v; }
};
template <> struct Cvt<bf16_t> {
  __device__ __forceinline__ static float to_f(bf16_t v) { return bf2f(v); }
  __device__ __forceinline__ static bf16_t from_f(float v) { return f2bf(v); }
};
template <> struct Cvt<f16_t> {
  __device__ __forceinline__ static float to_f(f16_t v) { return (float)__builtin_bit_cast(_Float16, v.bits); }
  __device__ __forceinline__ static f16_t from_f(float v) { return f16_t{(uint16_t)(pack_h2(v, 0.f) & 0xffffu)}; }
};

// ---------------------------------------------------------------- MFMA ----
// 32x32 output block, accumulator layout (CDNA3/CDNA4): lane l holds column
// l % 32; acc[4*i + j] is row 8*i + 4*(l / 32) + j.
__device__ __forceinline__ f32x16_t mfma32_bf16(const u32x4_t& a, const u32x4_t& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma32_f16(const u32x4_t& a, const u32x4_t& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c, 0,
                                                0, 0);
}
// The 16-bit operand types of the MFMA GEMMs: packing of two floats and the
// 32 x 32 x 16 product with float32 accumulation.
template <typename T>
struct Op16;
template <>
struct Op16<bf16_t> {
  __device__ __forceinline__ static uint32_t pack2(float lo, float hi) { return pack_bf2(lo, hi); }
  __device__ __forceinline__ static f32x16_t mma(const u32x4_t& a, const u32x4_t& b, f32x16_t c) {
    return mfma32_bf16(a, b, c);
  }
};
template <>
struct Op16<f16_t> {
  __device__ __forceinline__ static uint32_t pack2(float lo, float hi) { return pack_h2(lo, hi); }
  __device__ __forceinline__ static f32x16_t mma(const u32x4_t& a, const u32x4_t& b, f32x16_t c) {
    return mfma32_f16(a, b, c);
  }
};
__device__ __forceinline__ f32x16_t mfma32_f32(float a, float b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
// 16x16 output block: lane l holds column l % 16; acc[j] is row 4*(l / 16) + j.
__device__ __forceinline__ f32x4_t mfma16_bf16(const u32x4_t& a, const u32x4_t& b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma16_f32(float a, float b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ----------------------------------------------------------- reductions ----
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

// Deterministic block sum (fixed tree): every thread gets the result.
template <typename F>
__device__ F block_sum(F v, F* scratch /* >= blockDim/64 entries */) {
  v = wave_sum(v);
  const int w = threadIdx.x / WAVE, nw = blockDim.x / WAVE;
  __syncthreads();
  if ((threadIdx.x & (WAVE - 1)) == 0) scratch[w] = v;
  __syncthreads();
  F t = 0;
  for (int i = 0; i < nw; ++i) t += scratch[i];
  __syncthreads();
  return t;
}

// ------------------------------------------------------------ XCD remap ----
// Work-groups are dispatched round-robin over the 8 XCDs (id % 8). Remap so
// that consecutive logical ids run on the same XCD and share its L2.
__device__ __forceinline__ int xcd_remap(int pid, int total) {
  constexpr int NX = 8;
  const int xcd = pid % NX, local = pid / NX;
  const int base = total / NX, rem = total % NX;
  return xcd < rem ? xcd * (base + 1) + local : rem * (base + 1) + (xcd - rem) * base + local;
}

__host__ __device__ inline int cdiv(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ inline int round_up(int a, int b) { return cdiv(a, b) * b; }

}  // namespace sd
