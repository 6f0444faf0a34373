// Batched MFMA GEMM for gfx950 with fused epilogues.
//
//   C[b] (M x N) = A[b] (M x K) * op(B[b])
//
// A is row-major with K contiguous. B is either "NT" (row-major N x K, K
// contiguous; C = A B^T) or "NN" (row-major K x N, N contiguous; C = A B).
// All dimensions are multiples of the tile (the callers pad their buffers
// with zeros), so the kernel carries no bounds checks.
//
// Tile: 128 x 128 outputs per work-group of 256 threads (4 waves in 2 x 2,
// 64 x 64 per wave as 2 x 2 MFMA blocks of 32 x 32). One LDS stage holds 128
// bytes of K per tile row (64 bf16 or 32 fp32) in eight 16-byte chunks, rows
// padded to 144 bytes; two stages are double buffered.
//   bf16: v_mfma_f32_32x32x16_bf16, one 16-byte chunk per lane per MFMA.
//   fp32: v_mfma_f32_32x32x2f32, one 16-byte chunk feeds four MFMAs.
// Lane l (h = l / 32) reads chunk 2 g + h of its row for chunk-pair g, so A
// and B always agree on which k each lane supplies.
//
// NN staging transposes the B tile in registers (4 x 8 bf16 or 4 x 4 fp32
// blocks) so that LDS always holds K-contiguous rows.
//
// SYM mode computes only tiles with tile_m <= tile_n of a symmetric result
// and writes each value at (r, c) and (c, r); diagonal tiles write c >= r.
#pragma once

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "common.hpp"

namespace sd {

constexpr int G_ROWB = 144;                    // LDS bytes per tile row
constexpr int G_TILEB = 128 * G_ROWB;          // one 128-row operand tile

template <typename T> struct GemmK;
template <> struct GemmK<bf16_t> { static constexpr int BK = 64; };
template <> struct GemmK<f16_t> { static constexpr int BK = 64; };
template <> struct GemmK<float> { static constexpr int BK = 32; };

struct GemmShape {
  int M, N, K;
  int lda, ldb;
  long long sa, sb;   // batch strides in elements
  int batch;
  // Tile order (non-symmetric): 0 walks tile columns fastest, 1 tile rows
  // fastest. With few tile rows and a small A, rows-fastest makes the
  // work-groups that share a B column panel run together on one XCD, so the
  // panel comes from HBM once and from L2 after that.
  int m_fast = 0;
  // Tail split: space for partial accumulators that the caller may give
  // (part_cap floats); the launchers then cut the tiles of a last, partly
  // idle round of work-groups along K (tiles tail0 .. end, in `pieces`
  // pieces each; tail_pieces) and sum the pieces in a second launch.
  float* part = nullptr;
  long long part_cap = 0;
  int tail0 = 0, pieces = 0;
};

enum { EMIT_FULL = 0, EMIT_SYM_OFF = 1, EMIT_SYM_DIAG = 2 };

// ----------------------------------------------------- store helpers ------
// Four consecutive rows r0..r0+3 at column c (coalesced across lanes).
template <typename T>
__device__ __forceinline__ void st_col4(T* p, int ld, int r0, int c, const float v[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) p[(long long)(r0 + j) * ld + c] = Cvt<T>::from_f(v[j]);
}
// Row r, columns c0..c0+3 (c0 % 4 == 0).
__device__ __forceinline__ void st_row4(float* p, int ld, int r, int c0, const float v[4]) {
  *reinterpret_cast<float4*>(p + (long long)r * ld + c0) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void st_row4(bf16_t* p, int ld, int r, int c0, const float v[4]) {
  uint2 w;
  w.x = pack_bf2(v[0], v[1]);
  w.y = pack_bf2(v[2], v[3]);
  *reinterpret_cast<uint2*>(p + (long long)r * ld + c0) = w;
}

__device__ __forceinline__ void st_row4(f16_t* p, int ld, int r, int c0, const float v[4]) {
  uint2 w;
  w.x = pack_h2(v[0], v[1]);
  w.y = pack_h2(v[2], v[3]);
  *reinterpret_cast<uint2*>(p + (long long)r * ld + c0) = w;
}

// Store v (rows r0..r0+3, column c) into a symmetric-or-full matrix.
template <typename T>
__device__ __forceinline__ void emit4(T* p, int ld, int r0, int c, const float v[4], int mode) {
  if (mode == EMIT_FULL) {
    st_col4(p, ld, r0, c, v);
  } else if (mode == EMIT_SYM_OFF) {
    st_col4(p, ld, r0, c, v);
    st_row4(p, ld, c, r0, v);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = r0 + j;
      if (c >= r) {
        p[(long long)r * ld + c] = Cvt<T>::from_f(v[j]);
        p[(long long)c * ld + r] = Cvt<T>::from_f(v[j]);
      }
    }
  }
}

// ------------------------------------------------------- epilogues --------
// Gram: out32 = scale32 * C (fp32, optional), out16 = T16(scale16 * C)
// (optional; bf16 or fp16, rounded to nearest even). RW = false: stores from
// the MFMA layout (for tiles whose C tile does not fit in LDS).
// STREAM = false: the row-wise stores are ordinary stores (stream_outputs).
template <typename T16, bool RW = true, bool STREAM = true>
struct EpiGramT {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = RW;
  static constexpr bool HI_FROM_B = false;
  // Row-wise form (direct-to-LDS kernel): eight consecutive columns of row r.
  // The transposed (lower-triangle) copy gets out16 only (store8): out32 is
  // read back only at upper-triangle and diagonal-tile positions.
  __device__ void pre8(int, int, int, u32x4_t&, u32x4_t&) const {}
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t&, const u32x4_t&,
                         float (&mv)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
#pragma unroll
    for (int q = 0; q < 8; ++q) mv[q] = v[q] * scale16;
    if (out16) store8(b, r, c0, mv);
    if (out32) {
      const f32x4_t w0 = f32x4_t{v[0], v[1], v[2], v[3]} * scale32, w1 = f32x4_t{v[4], v[5], v[6], v[7]} * scale32;
      st16_pol<STREAM>(out32 + o, __builtin_bit_cast(u32x4_t, w0));
      st16_pol<STREAM>(out32 + o + 4, __builtin_bit_cast(u32x4_t, w1));
    }
  }
  __device__ void store8(int b, int r, int c0, const float (&v)[8]) const {
    if (out16)
      st16_pol<STREAM>(out16 + b * stride + (long long)r * ld + c0,
                       u32x4_t{Op16<T16>::pack2(v[0], v[1]), Op16<T16>::pack2(v[2], v[3]),
                               Op16<T16>::pack2(v[4], v[5]), Op16<T16>::pack2(v[6], v[7])});
  }
  float* out32;
  T16* out16;
  float scale32, scale16;
  long long stride;
  int ld;
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    if (out16) {
      float w[4] = {v[0] * scale16, v[1] * scale16, v[2] * scale16, v[3] * scale16};
      emit4(out16 + b * stride, ld, r0, c, w, mode);
    }
    if (out32) {
      float w[4] = {v[0] * scale32, v[1] * scale32, v[2] * scale32, v[3] * scale32};
      emit4(out32 + b * stride, ld, r0, c, w, mode);
    }
  }
  // Off-diagonal symmetric tiles, non-rowwise form (the kernel stages the
  // transposed copy through LDS): `direct` stores rows r0..r0+3 at column c
  // and hands back the values to mirror (here the raw product); `mirror8`
  // stores eight of them along row r from column c0.
  static constexpr bool MIRROR = !RW;
  __device__ void direct(int b, int r0, int c, const float v[4], float w[4]) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = v[j];
    operator()(b, r0, c, w, EMIT_FULL);
  }
  __device__ void mirror8(int b, int r, int c0, const float (&w)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
    if (out16)
      *reinterpret_cast<u32x4_t*>(out16 + o) =
          u32x4_t{Op16<T16>::pack2(w[0] * scale16, w[1] * scale16), Op16<T16>::pack2(w[2] * scale16, w[3] * scale16),
                  Op16<T16>::pack2(w[4] * scale16, w[5] * scale16), Op16<T16>::pack2(w[6] * scale16, w[7] * scale16)};
    if (out32) {
      *reinterpret_cast<f32x4_t*>(out32 + o) = f32x4_t{w[0], w[1], w[2], w[3]} * scale32;
      *reinterpret_cast<f32x4_t*>(out32 + o + 4) = f32x4_t{w[4], w[5], w[6], w[7]} * scale32;
    }
  }
};
using EpiGram = EpiGramT<bf16_t>;

// Polynomial in the Gram: out = bc * A32 + cc * C. STREAM = false: the
// 16-bit stores are ordinary stores (stream_outputs).
template <typename TO, bool STREAM = true>
struct EpiPoly {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = true;
  static constexpr bool HI_FROM_B = false;
  const float* a32;
  TO* out;
  float bc, cc;
  long long stride;
  int ld;
  // Row-wise form (direct-to-LDS kernel): eight consecutive columns of row r.
  // The A32 values are loaded before the main loop (pre8: columns c0..c0+3
  // in the first word group, c0+4..c0+7 in the second); the transposed copy
  // reuses the values (store8).
  __device__ void pre8(int b, int r, int c0, u32x4_t& h, u32x4_t& l) const {
    const long long o = b * stride + (long long)r * ld + c0;
    h = ld16(a32 + o);
    l = ld16(a32 + o + 4);
  }
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t& h, const u32x4_t& l,
                         float (&w)[8]) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[q] = bc * __uint_as_float(h[q]) + cc * v[q];
      w[q + 4] = bc * __uint_as_float(l[q]) + cc * v[q + 4];
    }
    store8(b, r, c0, w);
  }
  __device__ void store8(int b, int r, int c0, const float (&w)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
    if constexpr (sizeof(TO) == 2) {
      st16_pol<STREAM>(out + o, u32x4_t{Op16<TO>::pack2(w[0], w[1]), Op16<TO>::pack2(w[2], w[3]),
                                        Op16<TO>::pack2(w[4], w[5]), Op16<TO>::pack2(w[6], w[7])});
    } else {
      *reinterpret_cast<f32x4_t*>(out + o) = f32x4_t{w[0], w[1], w[2], w[3]};
      *reinterpret_cast<f32x4_t*>(out + o + 4) = f32x4_t{w[4], w[5], w[6], w[7]};
    }
  }
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    const float* a = a32 + b * stride;
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = bc * a[(long long)(r0 + j) * ld + c] + cc * v[j];
    emit4(out + b * stride, ld, r0, c, v, mode);
  }
};

// Iterate update: out = ac * X + C into the next padded iterate, or (final
// step) into the caller's output: rows < rows_valid, cols < cols_valid, in
// row-major [rows x cols] or transposed [cols x rows] with its own dtype.
// The X values are prefetched into registers before the main loop (pre), so
// their HBM reads overlap the products.
template <typename TX, typename TO>
struct EpiUpdate {
  static constexpr bool PRE = true;
  static constexpr bool ROWWISE = false;
  static constexpr bool HI_FROM_B = false;
  const TX* x;
  long long xstride;
  int ldx;
  float ac;
  TO* out;
  long long ostride;
  int ldo;
  int final_out;       // 0: padded iterate (same layout as x); 1: caller output
  int transpose_out;   // caller output is the transpose of the canonical iterate
  int rows_valid, cols_valid;
  bf16_t* out16;       // optional bf16 copy of the padded iterate (operand of the next products)
  __device__ float pre(int b, int r, int c) const { return Cvt<TX>::to_f(x[b * xstride + (long long)r * ldx + c]); }
  __device__ void apply(int b, int r0, int c, float v[4], int mode, const float* xv) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = ac * xv[j] + v[j];
    TO* ob = out + b * ostride;
    if (!final_out) {
      emit4(ob, ldo, r0, c, v, mode);
      if (out16) emit4(out16 + b * ostride, ldo, r0, c, v, mode);
      return;
    }
    if (c >= cols_valid) return;
    if (!transpose_out) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (r0 + j < rows_valid) ob[(long long)(r0 + j) * ldo + c] = Cvt<TO>::from_f(v[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (r0 + j < rows_valid) ob[(long long)c * ldo + r0 + j] = Cvt<TO>::from_f(v[j]);
    }
  }
};

// Full product scaled by a device scalar: out = (*scale) C, fp32; row-wise,
// or from the MFMA layout (RW = false).
template <bool RW = true>
struct EpiScaleStore {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = RW;
  static constexpr bool HI_FROM_B = false;
  float* out;
  const float* scale;
  long long stride;
  int ld;
  __device__ void pre8(int, int, int, u32x4_t&, u32x4_t&) const {}
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t&, const u32x4_t&,
                         float (&w)[8]) const {
    const float s = *scale;
#pragma unroll
    for (int q = 0; q < 8; ++q) w[q] = v[q] * s;
    store8(b, r, c0, w);
  }
  __device__ void store8(int b, int r, int c0, const float (&w)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
    *reinterpret_cast<f32x4_t*>(out + o) = f32x4_t{w[0], w[1], w[2], w[3]};
    *reinterpret_cast<f32x4_t*>(out + o + 4) = f32x4_t{w[4], w[5], w[6], w[7]};
  }
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    const float s = *scale;
    float w[4] = {v[0] * s, v[1] * s, v[2] * s, v[3] * s};
    emit4(out + b * stride, ld, r0, c, w, mode);
  }
};

// Iterate update of a symmetric filter (X and the polynomial in X commute,
// so X_next = ac X + B X is symmetric and computed on upper-triangle tiles):
// row-wise, out = ac * x + C in fp32 and its T16 copy (the next products'
// operand). The x values are loaded before the main loop (pre8).
template <typename T16>
struct EpiUpdateSym {
  static constexpr bool PRE = true;
  static constexpr bool ROWWISE = true;
  static constexpr bool HI_FROM_B = false;
  const float* x;
  float ac;
  float* out;
  T16* out16;
  long long stride;
  int ld;
  __device__ void pre8(int b, int r, int c0, u32x4_t& h, u32x4_t& l) const {
    const long long o = b * stride + (long long)r * ld + c0;
    h = ld16(x + o);
    l = ld16(x + o + 4);
  }
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t& h, const u32x4_t& l,
                         float (&w)[8]) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[q] = ac * __uint_as_float(h[q]) + v[q];
      w[q + 4] = ac * __uint_as_float(l[q]) + v[q + 4];
    }
    store8(b, r, c0, w);
  }
  __device__ void store8(int b, int r, int c0, const float (&w)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
    st16_nt(out + o, __builtin_bit_cast(u32x4_t, f32x4_t{w[0], w[1], w[2], w[3]}));
    st16_nt(out + o + 4, __builtin_bit_cast(u32x4_t, f32x4_t{w[4], w[5], w[6], w[7]}));
    st16_nt(out16 + o, u32x4_t{Op16<T16>::pack2(w[0], w[1]), Op16<T16>::pack2(w[2], w[3]),
                               Op16<T16>::pack2(w[4], w[5]), Op16<T16>::pack2(w[6], w[7])});
  }
  __device__ void operator()(int, int, int, float*, int) const {}
};

// EpiUpdateSym from the MFMA layout, for tiles whose C tile does not fit in
// LDS: x is read after the main loop (the long K loops this form serves
// leave that read negligible; a non-temporal load, as each value is read
// once), both outputs through emit4 (mirrored on off-diagonal tiles).
// STREAM: the fp32 output of off-diagonal tiles is written with streaming
// stores (stream_outputs: on outputs too large to stay in the last-level
// cache for the next step).
template <typename T16, bool STREAM = false>
struct EpiUpdateSymNR {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = false;
  static constexpr bool HI_FROM_B = false;
  const float* x;
  float ac;
  float* out;
  T16* out16;
  long long stride;
  int ld;
  __device__ void pre8(int, int, int, u32x4_t&, u32x4_t&) const {}
  __device__ void apply8(int, int, int, const float (&)[8], const u32x4_t&, const u32x4_t&, float (&)[8]) const {}
  __device__ void store8(int, int, int, const float (&)[8]) const {}
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    const float* xb = x + b * stride;
    float w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = ac * __builtin_nontemporal_load(&xb[(long long)(r0 + j) * ld + c]) + v[j];
    emit4(out + b * stride, ld, r0, c, w, mode);
    emit4(out16 + b * stride, ld, r0, c, w, mode);
  }
  // off-diagonal tiles: the transposed copy is staged through LDS (EpiGramT)
  static constexpr bool MIRROR = true;
  __device__ void direct(int b, int r0, int c, const float v[4], float w[4]) const {
    const float* xb = x + b * stride;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = ac * __builtin_nontemporal_load(&xb[(long long)(r0 + j) * ld + c]) + v[j];
    if constexpr (STREAM) {
      float* ob = out + b * stride;
#pragma unroll
      for (int j = 0; j < 4; ++j) __builtin_nontemporal_store(w[j], &ob[(long long)(r0 + j) * ld + c]);
    } else {
      st_col4(out + b * stride, ld, r0, c, w);
    }
    st_col4(out16 + b * stride, ld, r0, c, w);
  }
  __device__ void mirror8(int b, int r, int c0, const float (&w)[8]) const {
    const long long o = b * stride + (long long)r * ld + c0;
    st16_pol<STREAM>(out + o, __builtin_bit_cast(u32x4_t, f32x4_t{w[0], w[1], w[2], w[3]}));
    st16_pol<STREAM>(out + o + 4, __builtin_bit_cast(u32x4_t, f32x4_t{w[4], w[5], w[6], w[7]}));
    *reinterpret_cast<u32x4_t*>(out16 + o) =
        u32x4_t{Op16<T16>::pack2(w[0], w[1]), Op16<T16>::pack2(w[2], w[3]), Op16<T16>::pack2(w[4], w[5]),
                Op16<T16>::pack2(w[6], w[7])};
  }
};

// Iterate update with the bf16 iterate stored as hi = bf16(X) plus an e4m3
// residual byte (state_pack8 / state_value8): out = ac * X + C, written in the
// same form, or (final step) into the caller's output with the rules of
// EpiUpdate. hi is the product operand of the next step.
// Row-wise epilogue: the kernel hands it eight consecutive columns of one row
// (the accumulators pass through LDS), so global accesses are 16 bytes (hi)
// and 8 bytes (residuals) wide. The residuals are loaded before the main loop (pre8); hi is the
// product's B operand itself (X, K x N with K = the rows of the iterate), so
// the kernel copies it out of the LDS ring while the K steps that cover the
// tile's rows pass through (HI_FROM_B) instead of reading it again from HBM.
template <typename TO>
struct EpiUpdateHL {
  static constexpr bool PRE = true;
  static constexpr bool ROWWISE = true;
  static constexpr bool HI_FROM_B = true;
  const bf16_t* hi;
  const int8_t* lo;    // residual bytes, same element layout as hi
  long long xstride;
  int ldx;
  float ac;
  bf16_t* out_hi;      // next state (same layout as hi / lo)
  int8_t* out_lo;
  TO* out;             // final step: caller output
  long long ostride;
  int ldo;
  int final_out;
  int transpose_out;
  int rows_valid, cols_valid;
  // (the residual bytes are read once: a non-temporal load, which leaves the
  // caches to the operand tiles; 132.1 -> 129.6 us per launch at 24 x 768 x 3072)
  __device__ void pre8(int b, int r, int c0, u32x4_t&, u32x4_t& l) const {
    const u32x2_t w =
        __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(lo + b * xstride + (long long)r * ldx + c0));
    l = u32x4_t{w[0], w[1], 0u, 0u};
  }
  __device__ void apply8(int b, int r, int c0, const float (&acc)[8], const u32x4_t& h, const u32x4_t& l,
                         float (&)[8]) const {
    const uint32_t hw[4] = {h[0], h[1], h[2], h[3]};
    float v[8];
    state_value8(hw, l[0], l[1], v);
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = ac * v[q] + acc[q];
    if (!final_out) {
      uint32_t nh[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) nh[q] = pack_bf2(v[2 * q], v[2 * q + 1]);
      const long long o = b * xstride + (long long)r * ldx + c0;
      st16_nt(out_hi + o, u32x4_t{nh[0], nh[1], nh[2], nh[3]});
      st8_nt(out_lo + o, state_pack8(v, nh));
      return;
    }
    if (r >= rows_valid) return;
    TO* ob = out + b * ostride;
    if (!transpose_out) {
      if constexpr (sizeof(TO) == 2) {
        if (c0 + 8 <= cols_valid && (ldo & 7) == 0) {
          st16_nt(ob + (long long)r * ldo + c0,
               u32x4_t{pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]), pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7])});
          return;
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (c0 + q < cols_valid) ob[(long long)r * ldo + c0 + q] = Cvt<TO>::from_f(v[q]);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (c0 + q < cols_valid) ob[(long long)(c0 + q) * ldo + r] = Cvt<TO>::from_f(v[q]);
    }
  }
};

// Iterate update in transposed form: the kernel computes C^T = X^T B (B
// symmetric), so v[j] is element (c, r0 + j) of the new iterate: a lane owns
// four consecutive columns of one row and moves them as 16-byte vectors.
// out = ac * X + C, into the padded iterate (plus its bf16 copy), or (final
// step) the caller's output with the same rules as EpiUpdate.
template <typename TO>
struct EpiUpdateT {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = false;
  static constexpr bool HI_FROM_B = false;
  const float* x;
  long long xstride;
  int ldx;
  float ac;
  TO* out;
  long long ostride;
  int ldo;
  int final_out;
  int transpose_out;
  int rows_valid, cols_valid;
  bf16_t* out16;
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    const int row = c, col0 = r0;
    const f32x4_t xv = *reinterpret_cast<const f32x4_t*>(x + b * xstride + (long long)row * ldx + col0);
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = ac * xv[j] + v[j];
    TO* ob = out + b * ostride;
    if (!final_out) {
      st_row4(ob, ldo, row, col0, v);
      if (out16) st_row4(out16 + b * ostride, ldo, row, col0, v);
      return;
    }
    if (row >= rows_valid) return;
    if (!transpose_out) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (col0 + j < cols_valid) ob[(long long)row * ldo + col0 + j] = Cvt<TO>::from_f(v[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (col0 + j < cols_valid) ob[(long long)(col0 + j) * ldo + row] = Cvt<TO>::from_f(v[j]);
    }
  }
};

// Plain fp32 store of C.
struct EpiStore {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = false;
  static constexpr bool HI_FROM_B = false;
  float* out;
  long long stride;
  int ld;
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    emit4(out + b * stride, ld, r0, c, v, mode);
  }
};

// out = alpha x + C, alpha read from device memory (null: 1), plus an
// optional fp16 copy of alpha x in the same layout. x may alias out: each
// element of x is read before the main loop by the lane that later writes it.
struct EpiAxpyDev {
  static constexpr bool PRE = true;
  static constexpr bool ROWWISE = false;
  static constexpr bool HI_FROM_B = false;
  const float* x;
  const float* alpha;
  float* out;
  f16_t* xs16;
  int ld;
  __device__ float pre(int, int r, int c) const { return x[(long long)r * ld + c]; }
  __device__ void apply(int, int r0, int c, float v[4], int mode, const float* xv) const {
    const float a = alpha ? *alpha : 1.f;
    if (xs16) {
      float w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = a * xv[j];
      emit4(xs16, ld, r0, c, w, mode);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = fmaf(a, xv[j], v[j]);
    emit4(out, ld, r0, c, v, mode);
  }
};

// Plain fp32 store of C in the row-wise form (direct-to-LDS kernel).
struct EpiStoreRows {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = true;
  static constexpr bool HI_FROM_B = false;
  float* out;
  long long stride;
  int ld;
  __device__ void pre8(int, int, int, u32x4_t&, u32x4_t&) const {}
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t&, const u32x4_t&,
                         float (&)[8]) const {
    float* p = out + b * stride + (long long)r * ld + c0;
    *reinterpret_cast<f32x4_t*>(p) = f32x4_t{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4_t*>(p + 4) = f32x4_t{v[4], v[5], v[6], v[7]};
  }
};

// Product of a split-operand panel (the bf16 tall-skinny products of float32
// panels): the A operand holds panel row j < split twice, as hi in row j and
// lo in row split + j, and the whole M range is one tile. The kernel adds the
// partner row's values to every row below split (SPLIT), so output row j is
// the sum of the pair; rows split .. rows_out - 1 are written as zero and
// rows from rows_out on are not stored.
struct EpiStoreRowsSplit {
  static constexpr bool PRE = false;
  static constexpr bool ROWWISE = true;
  static constexpr bool HI_FROM_B = false;
  static constexpr bool SPLIT = true;
  float* out;
  long long stride;
  int ld;
  int split, rows_out;
  __device__ void pre8(int, int, int, u32x4_t&, u32x4_t&) const {}
  __device__ void apply8(int b, int r, int c0, const float (&v)[8], const u32x4_t&, const u32x4_t&,
                         float (&)[8]) const {
    if (r >= rows_out) return;
    float* p = out + b * stride + (long long)r * ld + c0;
    const bool keep = r < split;
    *reinterpret_cast<f32x4_t*>(p) = keep ? f32x4_t{v[0], v[1], v[2], v[3]} : f32x4_t{};
    *reinterpret_cast<f32x4_t*>(p + 4) = keep ? f32x4_t{v[4], v[5], v[6], v[7]} : f32x4_t{};
  }
};

// Epilogues that sum split row pairs declare SPLIT = true.
template <typename E, typename = void>
struct EpiSplit {
  static constexpr bool value = false;
};
template <typename E>
struct EpiSplit<E, std::void_t<decltype(E::SPLIT)>> {
  static constexpr bool value = E::SPLIT;
};

// Epilogues whose off-diagonal symmetric tiles take the LDS-staged transposed
// copy declare MIRROR = true (with `direct` and `mirror8`).
template <typename E, typename = void>
struct EpiMirror {
  static constexpr bool value = false;
};
template <typename E>
struct EpiMirror<E, std::void_t<decltype(E::MIRROR)>> {
  static constexpr bool value = E::MIRROR;
};

// ------------------------------------------------------- staging ----------
// Tile configuration: NWM x NWN waves, each computing WM x WN MFMA blocks of
// 32 x 32, so a work-group owns a (32 WM NWM) x (32 WN NWN) tile of C.
// STAGES = 2 double-buffers the LDS tiles (one barrier per K step); 1 keeps a
// single LDS buffer (two barriers per K step) so that two work-groups fit on
// a CU and one's epilogue overlaps the other's main loop.
// OCC: minimum waves per SIMD the register allocation must allow (0: the
// compiler's choice for the block size).
// BK: K step of the direct-to-LDS kernel (64 or 32; the register-staged
// kernel takes its K step from the element type).
template <int NWM_, int NWN_, int WM_, int WN_, int STAGES_ = 2, int OCC_ = 0, int BK_ = 64>
struct GemmCfg {
  static constexpr int NWM = NWM_, NWN = NWN_, WM = WM_, WN = WN_, STAGES = STAGES_, BK = BK_;
  static constexpr int OCC = OCC_ ? OCC_ : (64 * NWM_ * NWN_ + 255) / 256;
  static constexpr int BM = 32 * WM * NWM, BN = 32 * WN * NWN;
  static constexpr int NT = 64 * NWM * NWN;
};
using CfgTile128 = GemmCfg<2, 2, 2, 2>;          // 128 x 128, 256 threads
using CfgTile256 = GemmCfg<2, 4, 4, 2>;          // 256 x 256, 512 threads
// Single-stage tiles with registers capped for two work-groups per CU, so
// that one's epilogue (HBM traffic) overlaps the other's main loop.
using CfgTile256x128s = GemmCfg<2, 2, 4, 2, 1, 2>;   // 256 x 128, 256 threads
using CfgTile128s = GemmCfg<2, 2, 2, 2, 1, 2>;       // 128 x 128, 256 threads
// Direct-to-LDS kernel: 128 x 128, two-stage ring, two work-groups per CU.
using CfgDma128 = GemmCfg<2, 2, 2, 2, 2, 2>;
using CfgDma256 = GemmCfg<2, 4, 4, 2, 2, 2>;   // 256 x 256, eight waves, one work-group per CU

// Eight floats (two 16-byte words) rounded to eight 16-bit operands of type T.
template <typename T>
__device__ __forceinline__ u32x4_t pack8(const u32x4_t& a, const u32x4_t& b) {
  return u32x4_t{Op16<T>::pack2(__uint_as_float(a[0]), __uint_as_float(a[1])),
                 Op16<T>::pack2(__uint_as_float(a[2]), __uint_as_float(a[3])),
                 Op16<T>::pack2(__uint_as_float(b[0]), __uint_as_float(b[1])),
                 Op16<T>::pack2(__uint_as_float(b[2]), __uint_as_float(b[3]))};
}

// Rows x K tile with K contiguous in memory (the A operand, and B in NT form):
// ROWS rows of 8 LDS chunks of 16 bytes; chunk id = t + NT u -> row id / 8,
// chunk id % 8. An fp32 source feeding 16-bit MFMAs (bf16 or fp16) loads 32
// bytes per chunk and rounds them while writing LDS.
template <int ROWS, int NT, typename T, typename S>
struct RowStager {
  static constexpr bool CONV = sizeof(S) != sizeof(T);
  static constexpr int UNITS = ROWS * 8 / NT;
  static constexpr int LOADS = UNITS * (CONV ? 2 : 1);
  u32x4_t r[LOADS];
  __device__ __forceinline__ void load(const S* base, int ld, int row0, int k0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, row = id >> 3, ch = id & 7;
      const S* p = base + (long long)(row0 + row) * ld + k0 + ch * (CONV ? 8 : 16 / (int)sizeof(S));
      if constexpr (CONV) {
        r[2 * u] = ld16(p);
        r[2 * u + 1] = ld16(p + 4);
      } else {
        r[u] = ld16(p);
      }
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, row = id >> 3, ch = id & 7;
      if constexpr (CONV) st16(lds + row * G_ROWB + ch * 16, pack8<T>(r[2 * u], r[2 * u + 1]));
      else st16(lds + row * G_ROWB + ch * 16, r[u]);
    }
  }
};

// K x COLS tile with COLS contiguous in memory (B in NN form), transposed into
// LDS rows of K. A thread block covers 4 consecutive k and 8 (bf16 LDS) or 4
// (fp32 LDS) consecutive columns; block id = t + NT u -> kb = id % KB,
// nb = id / KB.
template <int COLS, int NT, typename T, typename S>
struct NNStager;

template <int COLS, int NT, typename S>
struct NNStager<COLS, NT, bf16_t, S> {       // 64 x COLS tile, bf16 LDS
  static constexpr bool CONV = sizeof(S) == 4;
  static constexpr int KB = 16;
  static constexpr int UNITS = KB * (COLS / 8) / NT;
  static constexpr int PER = CONV ? 8 : 4;    // 16-byte loads per unit
  u32x4_t r[UNITS * PER];
  __device__ __forceinline__ void load(const S* base, int ld, int k0, int n0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, kb = id % KB, nb = id / KB;
      const S* p = base + (long long)(k0 + 4 * kb) * ld + n0 + 8 * nb;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (CONV) {
          r[u * PER + 2 * i] = ld16(p + i * (long long)ld);
          r[u * PER + 2 * i + 1] = ld16(p + i * (long long)ld + 4);
        } else {
          r[u * PER + i] = ld16(p + i * (long long)ld);
        }
      }
    }
  }
  // 16-bit element c (0..7) of row i of unit u (bf16 source)
  __device__ __forceinline__ uint32_t half_bits(int u, int i, int c) const {
    const uint32_t w = r[u * PER + i][c >> 1];
    return (c & 1) ? (w >> 16) : (w & 0xffffu);
  }
  // fp32 element c (0..7) of row i of unit u (fp32 source)
  __device__ __forceinline__ float elem(int u, int i, int c) const {
    return __uint_as_float(r[u * PER + 2 * i + (c >> 2)][c & 3]);
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, kb = id % KB, nb = id / KB;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        u32x2_t v;
        if constexpr (CONV) {
          v = u32x2_t{pack_bf2(elem(u, 0, c), elem(u, 1, c)), pack_bf2(elem(u, 2, c), elem(u, 3, c))};
        } else {
          v = u32x2_t{half_bits(u, 0, c) | (half_bits(u, 1, c) << 16), half_bits(u, 2, c) | (half_bits(u, 3, c) << 16)};
        }
        *reinterpret_cast<u32x2_t*>(lds + (8 * nb + c) * G_ROWB + 8 * kb) = v;
      }
    }
  }
};

template <int COLS, int NT>
struct NNStager<COLS, NT, float, float> {    // 32 x COLS tile, fp32 LDS
  static constexpr int KB = 8;
  static constexpr int UNITS = KB * (COLS / 4) / NT;
  u32x4_t r[UNITS * 4];
  __device__ __forceinline__ void load(const float* base, int ld, int k0, int n0) {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, kb = id % KB, nb = id / KB;
      const float* p = base + (long long)(k0 + 4 * kb) * ld + n0 + 4 * nb;
#pragma unroll
      for (int i = 0; i < 4; ++i) r[u * 4 + i] = ld16(p + i * (long long)ld);
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int id = t + NT * u, kb = id % KB, nb = id / KB;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x4_t w = {r[u * 4][j], r[u * 4 + 1][j], r[u * 4 + 2][j], r[u * 4 + 3][j]};
        st16(lds + (4 * nb + j) * G_ROWB + 16 * kb, w);
      }
    }
  }
};

// ---------------------------------------------------------- compute -------
template <typename T, int WM, int WN>
__device__ __forceinline__ void tile_mma(const char* la, const char* lb, f32x16_t (&acc)[WM][WN], int wm,
                                         int wn, int lane) {
  const int r32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    u32x4_t a[WM], b[WN];
#pragma unroll
    for (int i = 0; i < WM; ++i) a[i] = ld16(la + (wm * WM * 32 + i * 32 + r32) * G_ROWB + (2 * g + h) * 16);
#pragma unroll
    for (int i = 0; i < WN; ++i) b[i] = ld16(lb + (wn * WN * 32 + i * 32 + r32) * G_ROWB + (2 * g + h) * 16);
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni) {
        if constexpr (sizeof(T) == 2) {
          acc[mi][ni] = Op16<T>::mma(a[mi], b[ni], acc[mi][ni]);
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t) acc[mi][ni] = mfma32_f32(u4f(a[mi], t), u4f(b[ni], t), acc[mi][ni]);
        }
      }
  }
}

// Upper-triangle tile index -> (tm, tn) with tm <= tn.
__device__ __forceinline__ void sym_tile(int t, int nt, int& tm, int& tn) {
  int m = 0;
  while (t >= nt - m) {
    t -= nt - m;
    ++m;
  }
  tm = m;
  tn = m + t;
}

// T: MFMA / LDS element type; SA, SB: element types of A and B in memory
// (fp32 sources feed bf16 MFMAs through rounding in the staging step).
// A_KN: A is stored K x M (M contiguous) and transposed while staging, as B
// is in NN form.
// Tail split (sh.pieces > 1): work-groups from sh.tail0 on each compute one
// K piece of a tile of the last round and store the accumulators to sh.part
// (piece u of tile t at unit (t - tail0) pieces + u, in the MFMA fragment
// layout as 16-byte groups of four accumulators, consecutive threads at
// consecutive groups); FIXUP launches one work-group per such tile, sums its
// pieces in piece order and runs the epilogue.
template <typename Cfg, typename T, typename SA, typename SB, bool A_KN, bool B_NN, bool SYM, typename Epi,
          bool FIXUP = false>
__global__ __attribute__((amdgpu_flat_work_group_size(1, Cfg::NT), amdgpu_waves_per_eu(Cfg::OCC))) void gemm_kernel(const SA* __restrict__ A, const SB* __restrict__ B,
                                                       GemmShape sh, Epi epi) {
  constexpr int BK = GemmK<T>::BK;
  constexpr int BM = Cfg::BM, BN = Cfg::BN, NT = Cfg::NT, WM = Cfg::WM, WN = Cfg::WN;
  constexpr int TA = BM * G_ROWB, TB = BN * G_ROWB, STAGE = TA + TB;
  static_assert(!SYM || BM == BN, "symmetric tiling needs square tiles");
  __shared__ __attribute__((aligned(16))) char lds[Cfg::STAGES * STAGE];
  const int tiles_m = sh.M / BM, tiles_n = sh.N / BN;
  const int per = SYM ? tiles_m * (tiles_m + 1) / 2 : tiles_m * tiles_n;
  int lid, piece = 0;
  bool tail = false;
  if constexpr (FIXUP) {
    lid = sh.tail0 + (int)blockIdx.x;
  } else if (sh.pieces > 1 && (int)blockIdx.x >= sh.tail0) {
    const int u = (int)blockIdx.x - sh.tail0;
    lid = sh.tail0 + u / sh.pieces;
    piece = u - (u / sh.pieces) * sh.pieces;
    tail = true;
  } else {
    lid = xcd_remap(blockIdx.x, sh.pieces > 1 ? sh.tail0 : per * sh.batch);
  }
  const int b = lid / per;
  int t = lid - b * per, tm, tn;
  if (SYM) {
    sym_tile(t, tiles_m, tm, tn);
  } else if (sh.m_fast) {
    tn = t / tiles_m;
    tm = t - tn * tiles_m;
  } else {
    tm = t / tiles_n;
    tn = t - tm * tiles_n;
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const SA* Ab = A + b * sh.sa;
  const SB* Bb = B + b * sh.sb;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int wm = wave / Cfg::NWN, wn = wave % Cfg::NWN;

  f32x16_t acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[i][j] = f32x16_t{};

  const int r32 = lane & 31, h = lane >> 5;
  // epilogue operands this lane will need, loaded before the main loop
  constexpr bool PRE = Epi::PRE;
  float px[PRE ? WM * WN * 16 : 1];
  if constexpr (PRE) {
    if (!tail) {
#pragma unroll
      for (int mi = 0; mi < WM; ++mi)
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              px[(mi * WN + ni) * 16 + 4 * i + j] =
                  epi.pre(b, m0 + wm * WM * 32 + mi * 32 + 8 * i + 4 * h + j, n0 + wn * WN * 32 + ni * 32 + r32);
    }
  }

  // the fragment layout of the partial accumulators: 16-byte groups of four
  // accumulators, consecutive threads at consecutive groups
  constexpr int TILE = BM * BN;
  auto part_at = [&](int mi, int ni, int q) { return (((mi * WN + ni) * 4 + q) * NT + (int)threadIdx.x) * 4; };
  if constexpr (FIXUP) {
    const float* src = sh.part + (long long)(lid - sh.tail0) * sh.pieces * TILE;
    for (int pc = 0; pc < sh.pieces; ++pc) {
      f32x4_t v[WM][WN][4];
#pragma unroll
      for (int mi = 0; mi < WM; ++mi)
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            v[mi][ni][q] = *reinterpret_cast<const f32x4_t*>(src + (long long)pc * TILE + part_at(mi, ni, q));
      // every load of the piece is issued before the first sum (left to
      // itself the scheduler interleaved loads, waits and sums, with two or
      // three loads in flight)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mi = 0; mi < WM; ++mi)
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[mi][ni][4 * q + j] += v[mi][ni][q][j];
    }
  } else {
    using AStager = typename std::conditional<A_KN, NNStager<BM, NT, T, SA>, RowStager<BM, NT, T, SA>>::type;
    using BStager = typename std::conditional<B_NN, NNStager<BN, NT, T, SB>, RowStager<BN, NT, T, SB>>::type;
    AStager sa;
    BStager sb;
    auto load_tiles = [&](int k0) {
      if constexpr (A_KN) sa.load(Ab, sh.lda, k0, m0);
      else sa.load(Ab, sh.lda, m0, k0);
      if constexpr (B_NN) sb.load(Bb, sh.ldb, k0, n0);
      else sb.load(Bb, sh.ldb, n0, k0);
    };
    const int nk = sh.K / BK;
    const int kb = tail ? piece * nk / sh.pieces : 0, ke = tail ? (piece + 1) * nk / sh.pieces : nk;
    load_tiles(kb * BK);
    if constexpr (Cfg::STAGES == 2) {
      sa.store(lds);
      sb.store(lds + TA);
      __syncthreads();
      for (int kt = kb; kt < ke; ++kt) {
        const int cur = (kt - kb) & 1;
        const bool more = kt + 1 < ke;
        if (more) load_tiles((kt + 1) * BK);
        tile_mma<T, WM, WN>(lds + cur * STAGE, lds + cur * STAGE + TA, acc, wm, wn, lane);
        if (more) {
          char* nxt = lds + (cur ^ 1) * STAGE;
          sa.store(nxt);
          sb.store(nxt + TA);
        }
        __syncthreads();
      }
    } else {
      for (int kt = kb; kt < ke; ++kt) {
        sa.store(lds);
        sb.store(lds + TA);
        __syncthreads();
        if (kt + 1 < ke) load_tiles((kt + 1) * BK);
        tile_mma<T, WM, WN>(lds, lds + TA, acc, wm, wn, lane);
        __syncthreads();
      }
    }
    if (tail) {
      float* dst = sh.part + (long long)((int)blockIdx.x - sh.tail0) * TILE;
#pragma unroll
      for (int mi = 0; mi < WM; ++mi)
#pragma unroll
        for (int ni = 0; ni < WN; ++ni)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f32x4_t*>(dst + part_at(mi, ni, q)) =
                f32x4_t{acc[mi][ni][4 * q], acc[mi][ni][4 * q + 1], acc[mi][ni][4 * q + 2], acc[mi][ni][4 * q + 3]};
      return;
    }
  }

  const int mode = SYM ? (tm == tn ? EMIT_SYM_DIAG : EMIT_SYM_OFF) : EMIT_FULL;
#pragma unroll
  for (int mi = 0; mi < WM; ++mi)
#pragma unroll
    for (int ni = 0; ni < WN; ++ni)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v[4] = {acc[mi][ni][4 * i], acc[mi][ni][4 * i + 1], acc[mi][ni][4 * i + 2],
                      acc[mi][ni][4 * i + 3]};
        const int r0 = m0 + wm * WM * 32 + mi * 32 + 8 * i + 4 * h;
        const int c = n0 + wn * WN * 32 + ni * 32 + r32;
        if constexpr (PRE) epi.apply(b, r0, c, v, mode, &px[(mi * WN + ni) * 16 + 4 * i]);
        else epi(b, r0, c, v, mode);
      }
}

// ------------------------------------------- bf16, direct-to-LDS loads -----
// gemm_dma_kernel: bf16 operands only. Tiles move from global memory into a
// ring of STAGES LDS buffers by global_load_lds_dwordx4 (no registers on
// the way), so STAGES - 1 K steps are in flight while one is multiplied;
// one barrier per K step.
//
// LDS layouts (16-byte chunks of 8 bf16; CH = BK / 8 chunks per K row):
//   row form (A, and B in NT form): row r holds K in CH chunks; logical chunk
//     c sits in slot c ^ ((r / (16 / CH)) % CH), so 16 consecutive rows read
//     at one logical chunk hit 16 distinct 16-byte bank groups.
//   NN form (B, K x N in memory): row k holds BN columns; chunk c (columns
//     8c..8c+7) sits in slot c ^ (4 (k & 3)), so the 32 lanes of one
//     transpose read (4 rows x 4 chunks each) meet 16 distinct 16-byte bank
//     groups. MFMA fragments are read with
//     the gfx950 LDS transpose read (ds_read_b64_tr_b16): a group of 16 lanes
//     whose lane i addresses row k0 + i / 4, columns n0 + 4 (i % 4) .. +3
//     receives in lane j the four values (k0 .. k0 + 3, n0 + j).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t* lds_bf16x4_ptr;

__device__ __forceinline__ u32x2_t lds_read_tr16(const char* p) {
  lds_bf16x4_ptr q = (lds_bf16x4_ptr)(p);
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4bf16(q));
}

// 16 bytes per lane from global memory straight into LDS at base + 16 lane
// (base wave-uniform), as inline assembly: the compiler then does not track
// the load as an LDS write, so it adds no wait on it before later LDS reads;
// the kernels order every such load with their own vmcnt waits and barriers.
// m0 carries the LDS address; nothing else in these kernels uses m0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(const void* g, char* base) {
  const unsigned off = (unsigned)(size_t)((__attribute__((address_space(3))) char*)base);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(__builtin_amdgcn_readfirstlane(off))
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int CH>
__device__ __forceinline__ int rowform_slot(int r, int c) {
  static_assert(CH == 4 || CH == 8, "K row of 4 or 8 chunks");
  return c ^ ((r / (16 / CH)) & (CH - 1));
}
__device__ __forceinline__ int nnform_slot(int k, int c) { return c ^ (4 * (k & 3)); }

// One K step of MFMAs from LDS: BK / 16 k-chunks, the fragments of chunk
// g + 1 read while chunk g's MFMAs issue.
template <int WM, int WN, int BN, int BK, bool B_NN>
__device__ __forceinline__ void load_frags_dma(const char* la, const char* lb, int g, u32x4_t (&a)[WM],
                                               u32x4_t (&b)[WN], int wm, int wn, int lane) {
  constexpr int RB = 2 * BK, CH = BK / 8;   // bytes and chunks per K row
  const int r32 = lane & 31, h = lane >> 5;
  const int q = lane >> 4, j = lane & 15;
  const int c = 2 * g + h;
#pragma unroll
  for (int i = 0; i < WM; ++i) {
    const int row = wm * WM * 32 + i * 32 + r32;
    a[i] = ld16(la + row * RB + (rowform_slot<CH>(row, c) << 4));
  }
  if constexpr (!B_NN) {
#pragma unroll
    for (int i = 0; i < WN; ++i) {
      const int row = wn * WN * 32 + i * 32 + r32;
      b[i] = ld16(lb + row * RB + (rowform_slot<CH>(row, c) << 4));
    }
  } else {
    const int k0 = 8 * (2 * g + (q >> 1)) + (j >> 2);
#pragma unroll
    for (int i = 0; i < WN; ++i) {
      const int col = wn * WN * 32 + i * 32 + 16 * (q & 1) + 4 * (j & 3);
      const int off = ((col & 7) << 1);
      const u32x2_t lo = lds_read_tr16(lb + k0 * (2 * BN) + (nnform_slot(k0, col >> 3) << 4) + off);
      const u32x2_t hi = lds_read_tr16(lb + (k0 + 4) * (2 * BN) + (nnform_slot(k0 + 4, col >> 3) << 4) + off);
      b[i] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    }
  }
}

template <typename T, int WM, int WN, int BN, int BK, bool B_NN>
__device__ __forceinline__ void tile_mma_dma(const char* la, const char* lb, f32x16_t (&acc)[WM][WN], int wm,
                                             int wn, int lane) {
  constexpr int G = BK / 16;
  u32x4_t a[2][WM], b[2][WN];
  load_frags_dma<WM, WN, BN, BK, B_NN>(la, lb, 0, a[0], b[0], wm, wn, lane);
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g + 1 < G)
      load_frags_dma<WM, WN, BN, BK, B_NN>(la, lb, g + 1, a[(g + 1) & 1], b[(g + 1) & 1], wm, wn, lane);
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni) acc[mi][ni] = Op16<T>::mma(a[g & 1][mi], b[g & 1][ni], acc[mi][ni]);
  }
}

// LDS bytes of gemm_dma_kernel: the ring, or the row-wise epilogue's C tile
// (rows padded to BN + 8 floats, so the two row groups a store instruction
// covers fall in different banks) where that is larger.
template <typename Cfg, bool ROWWISE, bool MIRROR = false>
struct DmaLds {
  static constexpr int RW_LD = Cfg::BN + 8;
  static constexpr int MIR_LD = Cfg::BM + 4;   // floats per row of the staged transposed half-tile
  static constexpr int RING = Cfg::STAGES * (Cfg::BM + Cfg::BN) * 2 * Cfg::BK;
  static constexpr int CT = ROWWISE ? Cfg::BM * RW_LD * 4 : 0;
  static constexpr int MIR = MIRROR ? (Cfg::BN / 2) * MIR_LD * 4 : 0;
  static constexpr int BYTES = RING > CT ? (RING > MIR ? RING : MIR) : (CT > MIR ? CT : MIR);
};

// One output tile (linear tile id lid over the batch). T: the 16-bit operand
// type (bf16 or fp16; the loads move bytes, only the MFMA differs).
// SPLIT (epilogues in the MFMA layout only): DMA_PIECE computes K steps
// kb .. ke - 1 and stores the accumulators to dst (the fragment layout of the
// register-staged kernel's tail split); DMA_FIXUP sums the tile's `pieces`
// partials at src in piece order and runs the epilogue.
enum { DMA_WHOLE = 0, DMA_PIECE = 1, DMA_FIXUP = 2 };
template <typename Cfg, typename T, bool B_NN, bool SYM, typename Epi, int SPLIT = DMA_WHOLE>
__device__ __forceinline__ void gemm_dma_tile(const T* __restrict__ A, const T* __restrict__ B,
                                              const GemmShape& sh, const Epi& epi, char* lds, int lid,
                                              int kb = 0, int ke = 0, float* dst = nullptr,
                                              const float* src = nullptr) {
  static_assert(SPLIT == DMA_WHOLE || !Epi::ROWWISE, "K pieces need an epilogue in the MFMA layout");
  constexpr int BK = Cfg::BK, RB = 2 * BK, CH = BK / 8, RPL = 1024 / RB;   // rows per 1 KB load
  constexpr int BM = Cfg::BM, BN = Cfg::BN, WM = Cfg::WM, WN = Cfg::WN, S = Cfg::STAGES;
  constexpr int NW = Cfg::NWM * Cfg::NWN;
  constexpr int A_BYTES = BM * RB, STAGE = (BM + BN) * RB;
  constexpr int LA = BM / RPL / NW;        // A load instructions (1 KB each) per wave per stage
  constexpr int LB = BN / RPL / NW;        // B: NT RPL rows each; NN 1 KB = 512 / BN K rows each
  constexpr int LT = LA + LB;
  static_assert(BK == 32 || BK == 64, "K step");
  static_assert(BM % (RPL * NW) == 0 && BN % (RPL * NW) == 0, "tile rows per wave");
  static_assert(S >= 2 && S <= 5 && LT * (S - 2) < 64, "stages");
  static_assert(!SYM || BM == BN, "symmetric tiling needs square tiles");
  constexpr int RW_LD = DmaLds<Cfg, Epi::ROWWISE>::RW_LD;

  const int tiles_m = sh.M / BM, tiles_n = sh.N / BN;
  const int per = SYM ? tiles_m * (tiles_m + 1) / 2 : tiles_m * tiles_n;
  const int b = lid / per;
  int t = lid - b * per, tm, tn;
  if (SYM) {
    sym_tile(t, tiles_m, tm, tn);
  } else if (sh.m_fast) {
    tn = t / tiles_m;
    tm = t - tn * tiles_m;
  } else {
    tm = t / tiles_n;
    tn = t - tm * tiles_n;
  }
  const int m0 = tm * BM, n0 = tn * BN;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int wm = wave / Cfg::NWN, wn = wave % Cfg::NWN;
  const int r32 = lane & 31, h = lane >> 5;

  // Epilogue operands this lane will need, loaded before the main loop: in
  // the MFMA layout (PRE), or 8-column row chunks (ROWWISE: chunk u of thread
  // t is element group t + NT u of the tile, row = group / (BN / 8)).
  constexpr bool PRE = Epi::PRE && !Epi::ROWWISE;
  constexpr bool ROWWISE = Epi::ROWWISE;
  constexpr int RW_CH = BM * BN / 8 / Cfg::NT;     // row chunks per thread
  float px[PRE ? WM * WN * 16 : 1];
  u32x4_t rw_h[ROWWISE ? RW_CH : 1], rw_l[ROWWISE ? RW_CH : 1];
  if constexpr (PRE && SPLIT != DMA_PIECE) {
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            px[(mi * WN + ni) * 16 + 4 * i + jj] =
                epi.pre(b, m0 + wm * WM * 32 + mi * 32 + 8 * i + 4 * h + jj, n0 + wn * WN * 32 + ni * 32 + r32);
  }
  if constexpr (ROWWISE) {
#pragma unroll
    for (int u = 0; u < RW_CH; ++u) {
      const int e = threadIdx.x + Cfg::NT * u;
      epi.pre8(b, m0 + e / (BN / 8), n0 + 8 * (e % (BN / 8)), rw_h[u], rw_l[u]);
    }
  }

  // per-lane global sources (at k = 0) and wave-uniform LDS offsets
  const T* ga[LA];
  int la_off[LA];
#pragma unroll
  for (int u = 0; u < LA; ++u) {
    const int qi = wave + NW * u;
    const int row = RPL * qi + lane / CH;
    const int ch = rowform_slot<CH>(row, lane % CH);   // slot -> logical chunk (xor is its own inverse)
    ga[u] = A + b * sh.sa + (long long)(m0 + row) * sh.lda + 8 * ch;
    la_off[u] = 1024 * qi;
  }
  const T* gb[LB];
  int lb_off[LB];
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const int qi = wave + NW * u;
    if constexpr (!B_NN) {
      const int row = RPL * qi + lane / CH;
      const int ch = rowform_slot<CH>(row, lane % CH);
      gb[u] = B + b * sh.sb + (long long)(n0 + row) * sh.ldb + 8 * ch;
    } else {
      constexpr int CPR = BN / 8;            // chunks per LDS row
      static_assert(CPR >= 16, "the NN swizzle needs rows of at least 16 chunks");
      constexpr int RPI = 64 / CPR;          // rows per load instruction
      const int k = RPI * qi + lane / CPR;
      const int ch = nnform_slot(k, lane % CPR);
      gb[u] = B + b * sh.sb + (long long)k * sh.ldb + n0 + 8 * ch;
    }
    lb_off[u] = A_BYTES + 1024 * qi;
  }
  const long long a_step = BK, b_step = B_NN ? (long long)BK * sh.ldb : (long long)BK;

  auto issue = [&](int slot, int kt) {
    char* base = lds + slot * STAGE;
#pragma unroll
    for (int u = 0; u < LA; ++u) lds_dma16(ga[u] + kt * a_step, base + la_off[u]);
#pragma unroll
    for (int u = 0; u < LB; ++u) lds_dma16(gb[u] + kt * b_step, base + lb_off[u]);
  };

  f32x16_t acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int jj = 0; jj < WN; ++jj) acc[i][jj] = f32x16_t{};

  // K steps k0 .. k0 + nk - 1 (all of them for a whole tile)
  const int k0 = SPLIT == DMA_PIECE ? kb : 0;
  const int nk = SPLIT == DMA_PIECE ? ke - kb : (SPLIT == DMA_FIXUP ? 0 : sh.K / BK);
  if constexpr (SPLIT == DMA_FIXUP) {
    // a piece's loads in groups of MH fragment rows (the accumulators and
    // one group's values fit the registers), all of a group's loads before
    // its sums
    constexpr int TILE = BM * BN, MH = WM > 2 ? WM / 2 : WM;
    for (int pc = 0; pc < sh.pieces; ++pc) {
#pragma unroll
      for (int m2 = 0; m2 < WM; m2 += MH) {
        f32x4_t v[MH][WN][4];
#pragma unroll
        for (int mi = 0; mi < MH; ++mi)
#pragma unroll
          for (int ni = 0; ni < WN; ++ni)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              v[mi][ni][q] = *reinterpret_cast<const f32x4_t*>(
                  src + (long long)pc * TILE + ((((m2 + mi) * WN + ni) * 4 + q) * Cfg::NT + (int)threadIdx.x) * 4);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int mi = 0; mi < MH; ++mi)
#pragma unroll
          for (int ni = 0; ni < WN; ++ni)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[m2 + mi][ni][4 * q + j] += v[mi][ni][q][j];
      }
    }
  }
#pragma unroll
  for (int s0 = 0; s0 < S - 1; ++s0)
    if (s0 < nk) issue(s0, k0 + s0);
  for (int i = 0; i < nk; ++i) {
    const int kt = k0 + i;
    // stage i has landed once at most the later stages' loads are pending
    const int later = nk - 1 - i < S - 2 ? nk - 1 - i : S - 2;
    if constexpr (S >= 5) {
      if (later >= 3) wait_vmcnt<LT * 3>();
      else if (later == 2) wait_vmcnt<LT * 2>();
      else if (later == 1) wait_vmcnt<LT>();
      else wait_vmcnt<0>();
    } else if constexpr (S == 4) {
      if (later >= 2) wait_vmcnt<LT * 2>();
      else if (later == 1) wait_vmcnt<LT>();
      else wait_vmcnt<0>();
    } else if constexpr (S == 3) {
      if (later >= 1) wait_vmcnt<LT>();
      else wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_barrier();
    if (i + S - 1 < nk) issue((i + S - 1) % S, kt + S - 1);
    const char* base = lds + (i % S) * STAGE;
    if constexpr (Epi::HI_FROM_B) {
      // rows [kt BK, kt BK + BK) of the B operand are rows of this tile's
      // output when they fall in [m0, m0 + BM): copy the epilogue's chunks
      static_assert(B_NN && !SYM && ROWWISE, "hi from B needs the update's layout");
      const int kb = kt * BK - m0;
      if (kb >= 0 && kb < BM) {
#pragma unroll
        for (int u = 0; u < RW_CH; ++u) {
          const int e = threadIdx.x + Cfg::NT * u;
          const int k = e / (BN / 8) - kb;
          if (k >= 0 && k < BK)
            rw_h[u] = ld16(base + A_BYTES + k * (2 * BN) + (nnform_slot(k, e % (BN / 8)) << 4));
        }
      }
    }
    tile_mma_dma<T, WM, WN, BN, BK, B_NN>(base, base + A_BYTES, acc, wm, wn, lane);
  }
  if constexpr (SPLIT == DMA_PIECE) {
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<f32x4_t*>(dst + (((mi * WN + ni) * 4 + q) * Cfg::NT + (int)threadIdx.x) * 4) =
              f32x4_t{acc[mi][ni][4 * q], acc[mi][ni][4 * q + 1], acc[mi][ni][4 * q + 2], acc[mi][ni][4 * q + 3]};
    return;
  }

  if constexpr (ROWWISE) {
    // accumulators -> LDS (row pitch RW_LD floats) -> 8-column row chunks.
    // Symmetric tiling: a diagonal tile takes C[r][c] for c >= r and C[c][r]
    // below (so the result is exactly symmetric); an off-diagonal tile also
    // writes its transpose at (n0 + c, m0 + r).
    float* ct = reinterpret_cast<float*>(lds);
    __syncthreads();
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            ct[(wm * WM * 32 + mi * 32 + 8 * i + 4 * h + jj) * RW_LD + wn * WN * 32 + ni * 32 + r32] =
                acc[mi][ni][4 * i + jj];
    __syncthreads();
    const bool diag = SYM && tm == tn;
    float mv[RW_CH][8];   // values of the transposed copy (symmetric tilings)
#pragma unroll
    for (int u = 0; u < RW_CH; ++u) {
      const int e = threadIdx.x + Cfg::NT * u;
      const int r = e / (BN / 8), c8 = 8 * (e % (BN / 8));
      const f32x4_t a0 = *reinterpret_cast<const f32x4_t*>(ct + r * RW_LD + c8);
      const f32x4_t a1 = *reinterpret_cast<const f32x4_t*>(ct + r * RW_LD + c8 + 4);
      float av[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
      if constexpr (EpiSplit<Epi>::value) {
        // one M tile (m0 = 0): row r's partner r + split is in this tile
        if (r < epi.split) {
#pragma unroll
          for (int q = 0; q < 8; ++q) av[q] += ct[(r + epi.split) * RW_LD + c8 + q];
        }
      }
      if (diag) {
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (c8 + q < r) av[q] = ct[(c8 + q) * RW_LD + r];
      }
      epi.apply8(b, m0 + r, n0 + c8, av, rw_h[u], rw_l[u], mv[u]);
    }
    if constexpr (SYM) {
      if (!diag) {
        // the values to mirror go back into the C tile, then out transposed
        __syncthreads();
#pragma unroll
        for (int u = 0; u < RW_CH; ++u) {
          const int e = threadIdx.x + Cfg::NT * u;
          const int r = e / (BN / 8), c8 = 8 * (e % (BN / 8));
          *reinterpret_cast<f32x4_t*>(ct + r * RW_LD + c8) = f32x4_t{mv[u][0], mv[u][1], mv[u][2], mv[u][3]};
          *reinterpret_cast<f32x4_t*>(ct + r * RW_LD + c8 + 4) = f32x4_t{mv[u][4], mv[u][5], mv[u][6], mv[u][7]};
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < RW_CH; ++u) {
          const int e = threadIdx.x + Cfg::NT * u;
          const int c = e / (BM / 8), r8 = 8 * (e % (BM / 8));
          float av[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) av[q] = ct[(r8 + q) * RW_LD + c];
          epi.store8(b, n0 + c, m0 + r8, av);
        }
      }
    }
  } else {
    const int mode = SYM ? (tm == tn ? EMIT_SYM_DIAG : EMIT_SYM_OFF) : EMIT_FULL;
    if constexpr (SYM && EpiMirror<Epi>::value) {
      if (mode == EMIT_SYM_OFF) {
        // the transposed copy goes through LDS, half the tile's columns at a
        // time, so that it leaves as 32-byte row chunks instead of scattered
        // 16-byte pieces. A wave's columns lie in one half: in that half's
        // pass it stores its own positions straight from the MFMA layout
        // (rows r0..r0+3 at column c: coalesced across lanes) and puts the
        // same values, transposed, into LDS; then every wave writes rows of
        // the staged block.
        constexpr int ML = DmaLds<Cfg, false, true>::MIR_LD, HC = BN / 2;
        static_assert(HC % (WN * 32) == 0, "a wave's columns within one half");
        float* lt = reinterpret_cast<float*>(lds);
        const int wh = (wn * WN * 32) / HC;   // the half holding this wave's columns
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          __syncthreads();   // the ring (or the previous half) is no longer read
          if (wh == half) {
#pragma unroll
            for (int mi = 0; mi < WM; ++mi) {
#pragma unroll
              for (int ni = 0; ni < WN; ++ni)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  const int rl = wm * WM * 32 + mi * 32 + 8 * i + 4 * h, cl = wn * WN * 32 + ni * 32 + r32;
                  const float v[4] = {acc[mi][ni][4 * i], acc[mi][ni][4 * i + 1], acc[mi][ni][4 * i + 2],
                                      acc[mi][ni][4 * i + 3]};
                  float w[4];
                  epi.direct(b, m0 + rl, n0 + cl, v, w);
                  *reinterpret_cast<f32x4_t*>(lt + (cl - half * HC) * ML + rl) = f32x4_t{w[0], w[1], w[2], w[3]};
                }
              // the epilogue's own loads one MFMA row of blocks at a time:
              // all of them next to the live accumulators spilled registers
              __builtin_amdgcn_sched_barrier(0);
            }
          }
          __syncthreads();
          for (int q = (int)threadIdx.x; q < HC * (BM / 8); q += Cfg::NT) {
            const int row = q / (BM / 8), c8 = (q - row * (BM / 8)) * 8;
            const f32x4_t a0 = *reinterpret_cast<const f32x4_t*>(lt + row * ML + c8);
            const f32x4_t a1 = *reinterpret_cast<const f32x4_t*>(lt + row * ML + c8 + 4);
            const float w8[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
            epi.mirror8(b, n0 + half * HC + row, m0 + c8, w8);
          }
        }
        return;
      }
    }
#pragma unroll
    for (int mi = 0; mi < WM; ++mi)
#pragma unroll
      for (int ni = 0; ni < WN; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v[4] = {acc[mi][ni][4 * i], acc[mi][ni][4 * i + 1], acc[mi][ni][4 * i + 2],
                        acc[mi][ni][4 * i + 3]};
          const int r0 = m0 + wm * WM * 32 + mi * 32 + 8 * i + 4 * h;
          const int c = n0 + wn * WN * 32 + ni * 32 + r32;
          if constexpr (PRE) epi.apply(b, r0, c, v, mode, &px[(mi * WN + ni) * 16 + 4 * i]);
          else epi(b, r0, c, v, mode);
        }
  }
}

// One work-group per tile (xcd_remap gives each XCD a contiguous range of
// tiles, so work-groups that share operand panels share an L2). A variant
// that walked several tiles per work-group measured no faster and needed
// about 20-100 more VGPRs.
template <typename Cfg, bool B_NN, bool SYM, typename Epi, typename T, int SPLIT = DMA_WHOLE>
__global__ __attribute__((amdgpu_flat_work_group_size(1, Cfg::NT), amdgpu_waves_per_eu(Cfg::OCC))) void
gemm_dma_kernel(const T* __restrict__ A, const T* __restrict__ B, GemmShape sh, Epi epi) {
  __shared__ __attribute__((aligned(1024))) char lds[DmaLds<Cfg, Epi::ROWWISE, SYM && EpiMirror<Epi>::value>::BYTES];
  const int tm = sh.M / Cfg::BM, tn = sh.N / Cfg::BN;
  const int total = (SYM ? tm * (tm + 1) / 2 : tm * tn) * sh.batch;
  constexpr long long TILE = (long long)Cfg::BM * Cfg::BN;
  if constexpr (SPLIT == DMA_FIXUP) {
    const int u = (int)blockIdx.x;   // tile tail0 + u
    gemm_dma_tile<Cfg, T, B_NN, SYM, Epi, DMA_FIXUP>(A, B, sh, epi, lds, sh.tail0 + u, 0, 0, nullptr,
                                                     sh.part + (long long)u * sh.pieces * TILE);
  } else if constexpr (SPLIT == DMA_PIECE) {
    // whole tiles 0 .. tail0 - 1, then the pieces of the tail tiles
    if ((int)blockIdx.x < sh.tail0) {
      gemm_dma_tile<Cfg, T, B_NN, SYM, Epi>(A, B, sh, epi, lds, xcd_remap(blockIdx.x, sh.tail0));
      return;
    }
    const int u = (int)blockIdx.x - sh.tail0, tile = u / sh.pieces, piece = u - tile * sh.pieces;
    const int nk = sh.K / Cfg::BK;
    gemm_dma_tile<Cfg, T, B_NN, SYM, Epi, DMA_PIECE>(A, B, sh, epi, lds, sh.tail0 + tile, piece * nk / sh.pieces,
                                                     (piece + 1) * nk / sh.pieces, sh.part + (long long)u * TILE);
  } else {
    gemm_dma_tile<Cfg, T, B_NN, SYM, Epi>(A, B, sh, epi, lds, xcd_remap(blockIdx.x, total));
  }
}

// Work-groups of `kern` (nt threads) resident on the current device at once:
// CUs x work-groups per CU, cached per device (0 when the runtime cannot tell).
template <typename K>
inline int gemm_slots(K kern, int nt, std::atomic<int> (&cache)[16]) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
  if (dev < 16) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, nt, 0) != hipSuccess) return 0;
  const int slots = cus * per_cu;
  if (dev < 16) cache[dev].store(slots, std::memory_order_relaxed);
  return slots;
}

// Pieces for a last round of tiles: with `slots` work-groups resident at once
// and a last round of rem = blocks % slots tiles, the number p of K pieces per
// tile (2 .. 16, at most the K steps, bounded by the caller's space for
// partials) for which the pieces' rounds, ceil(rem p / slots) / p of a
// whole-tile round, take least time, if that is at most 0.8 of a round; 0
// otherwise (no cut).
inline int tail_pieces(long long blocks, int slots, int nk, long long part_cap, long long tile) {
  if (slots <= 0 || blocks < slots) return 0;
  const long long rem = blocks % slots;
  if (rem == 0) return 0;
  int best = 0;
  double best_t = 0.8;
  for (int p = 2; p <= 16 && p <= nk; ++p) {
    if (rem * p * tile > part_cap) break;
    const double t = (double)((rem * p + slots - 1) / slots) / p;
    if (t < best_t - 1e-9) {
      best_t = t;
      best = p;
    }
  }
  return best;
}

template <typename Cfg, bool B_NN, bool SYM, typename Epi, typename T>
void launch_gemm_dma(const T* A, const T* B, const GemmShape& sh, const Epi& epi, hipStream_t stream) {
  static_assert(sizeof(T) == 2, "16-bit operands");
  const int tm = sh.M / Cfg::BM, tn = sh.N / Cfg::BN;
  const long long per = SYM ? (long long)tm * (tm + 1) / 2 : (long long)tm * tn;
  const long long blocks = per * sh.batch;
  if (blocks <= 0) return;
  GemmShape s2 = sh;
  s2.tail0 = 0;
  s2.pieces = 0;
  if constexpr (!Epi::ROWWISE) {
    if (sh.part) {
      static std::atomic<int> slots_cache[16];
      const int slots = gemm_slots(gemm_dma_kernel<Cfg, B_NN, SYM, Epi, T>, Cfg::NT, slots_cache);
      const int pieces = tail_pieces(blocks, slots, sh.K / Cfg::BK, sh.part_cap, (long long)Cfg::BM * Cfg::BN);
      if (pieces) {
        const long long rem = blocks % slots;
        s2.tail0 = (int)(blocks - rem);
        s2.pieces = pieces;
        hipLaunchKernelGGL((gemm_dma_kernel<Cfg, B_NN, SYM, Epi, T, DMA_PIECE>),
                           dim3((unsigned)(blocks - rem + rem * pieces)), dim3(Cfg::NT), 0, stream, A, B, s2, epi);
        hipLaunchKernelGGL((gemm_dma_kernel<Cfg, B_NN, SYM, Epi, T, DMA_FIXUP>), dim3((unsigned)rem),
                           dim3(Cfg::NT), 0, stream, A, B, s2, epi);
        return;
      }
    }
  }
  hipLaunchKernelGGL((gemm_dma_kernel<Cfg, B_NN, SYM, Epi, T>), dim3((unsigned)blocks), dim3(Cfg::NT), 0, stream, A,
                     B, s2, epi);
}

// Store policy of an epilogue whose outputs the next launch reads at once
// (the Gram's copies for the polynomial, the polynomial's B for the update):
// ordinary stores leave them in the 256 MB last-level cache for that reader
// when they fit in half of it (on the 24 x 768 x 3072 Muon filter, 84 MB of
// Gram copies and 28 MB of B: 1.496 -> 1.476 ms per call, the Gram 72.7 ->
// 69.3 us and the polynomial 33.0 -> 31.4 us per launch); larger outputs
// (the 1280-wide groups' 470-940 MB) are streamed as before.
inline bool stream_outputs(long long bytes) { return bytes > (128ll << 20); }

// The same epilogue with ordinary stores.
template <typename T16, bool RW>
EpiGramT<T16, RW, false> cached_stores(const EpiGramT<T16, RW, true>& e) {
  EpiGramT<T16, RW, false> r{};
  r.out32 = e.out32;
  r.out16 = e.out16;
  r.scale32 = e.scale32;
  r.scale16 = e.scale16;
  r.stride = e.stride;
  r.ld = e.ld;
  return r;
}
template <typename TO>
EpiPoly<TO, false> cached_stores(const EpiPoly<TO, true>& e) {
  return EpiPoly<TO, false>{e.a32, e.out, e.bc, e.cc, e.stride, e.ld};
}

// Host launcher (errors surface through hipGetLastError at the end of a call).
// M, N must be multiples of the tile and K of the K step.
template <typename Cfg, typename T, bool B_NN, bool SYM, bool A_KN = false, typename SA, typename SB, typename Epi>
void launch_gemm(const SA* A, const SB* B, const GemmShape& sh, const Epi& epi, hipStream_t stream) {
  const int tm = sh.M / Cfg::BM, tn = sh.N / Cfg::BN;
  const long long per = SYM ? (long long)tm * (tm + 1) / 2 : (long long)tm * tn;
  const long long blocks = per * sh.batch;
  if (blocks <= 0) return;
  auto kern = gemm_kernel<Cfg, T, SA, SB, A_KN, B_NN, SYM, Epi>;
  GemmShape s2 = sh;
  s2.tail0 = 0;
  s2.pieces = 0;
  if (sh.part) {
    // a last round of at most half the resident work-groups: its tiles cut
    // along K (tail_pieces)
    static std::atomic<int> slots_cache[16];
    const int slots = gemm_slots(kern, Cfg::NT, slots_cache);
    const int pieces = tail_pieces(blocks, slots, sh.K / GemmK<T>::BK, sh.part_cap, (long long)Cfg::BM * Cfg::BN);
    if (pieces) {
      const long long rem = blocks % slots;
      s2.tail0 = (int)(blocks - rem);
      s2.pieces = pieces;
      hipLaunchKernelGGL(kern, dim3((unsigned)(blocks - rem + rem * pieces)), dim3(Cfg::NT), 0, stream, A, B, s2,
                         epi);
      hipLaunchKernelGGL((gemm_kernel<Cfg, T, SA, SB, A_KN, B_NN, SYM, Epi, true>), dim3((unsigned)rem),
                         dim3(Cfg::NT), 0, stream, A, B, s2, epi);
      return;
    }
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(Cfg::NT), 0, stream, A, B, s2, epi);
}

}  // namespace sd
