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

// ------------------------------------------------- iterate state ----------
// The bf16 iterate is stored as hi = bf16(x) plus an 8-bit residual q in
// units of 2^-8 ulp(hi): q = clamp(rint((x - hi) 2^(142 - E)), -127, 127) for
// the (bf16 = fp32) exponent field E of hi, E taken as 1 for zero and
// subnormals, and read back as hi + q 2^(E - 142). The scalings are exact.
__device__ __forceinline__ int state_exp(float h) {
  const int f = (int)((__float_as_uint(h) >> 23) & 0xFFu);
  return f > 0 ? f : 1;
}
__device__ __forceinline__ int state_q8(float x, float h) {
  float t = __builtin_rintf(__builtin_amdgcn_ldexpf(x - h, 142 - state_exp(h)));
  t = fminf(fmaxf(t, -127.f), 127.f);
  return (int)t;
}
__device__ __forceinline__ float state_value(float h, int q) {
  return h + __builtin_amdgcn_ldexpf((float)q, state_exp(h) - 142);
}
// 8 residuals <-> 8 bytes
__device__ __forceinline__ u32x2_t pack_q8(const int (&q)[8]) {
  u32x2_t w;
#pragma unroll
  for (int i = 0; i < 2; ++i)
    w[i] = (uint32_t)(q[4 * i] & 0xFF) | ((uint32_t)(q[4 * i + 1] & 0xFF) << 8) |
           ((uint32_t)(q[4 * i + 2] & 0xFF) << 16) | ((uint32_t)(q[4 * i + 3] & 0xFF) << 24);
  return w;
}
__device__ __forceinline__ int unpack_q8(const u32x2_t& w, int i) {
  return (int)(int8_t)((w[i >> 2] >> (8 * (i & 3))) & 0xFFu);
}

// Component i (a compile-time constant after unrolling) of a 16-byte value.
__device__ __forceinline__ uint32_t u4c(const u32x4_t& u, int i) { return u[i]; }
__device__ __forceinline__ float u4f(const u32x4_t& u, int i) { return __uint_as_float(u[i]); }
__device__ __forceinline__ u32x4_t ld16(const void* p) { return *reinterpret_cast<const u32x4_t*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4_t& v) { *reinterpret_cast<u32x4_t*>(p) = v; }

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

// ---------------------------------------------------------------- MFMA ----
// 32x32 output block, accumulator layout (CDNA3/CDNA4): lane l holds column
// l % 32; acc[4*i + j] is row 8*i + 4*(l / 32) + j.
__device__ __forceinline__ f32x16_t mfma32_bf16(const u32x4_t& a, const u32x4_t& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
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
