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

#include "common.hpp"

namespace sd {

constexpr int G_BM = 128, G_BN = 128, G_THREADS = 256;
constexpr int G_ROWB = 144;                    // LDS bytes per tile row
constexpr int G_TILEB = 128 * G_ROWB;          // one operand tile

template <typename T> struct GemmK;
template <> struct GemmK<bf16_t> { static constexpr int BK = 64; };
template <> struct GemmK<float> { static constexpr int BK = 32; };

struct GemmShape {
  int M, N, K;
  int lda, ldb;
  long long sa, sb;   // batch strides in elements
  int batch;
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
// Gram: out32 = scale32 * C (fp32, optional), out16 = bf16(scale16 * C)
// (optional).
struct EpiGram {
  float* out32;
  bf16_t* out16;
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
};

// Polynomial in the Gram: out = bc * A32 + cc * C.
template <typename TO>
struct EpiPoly {
  const float* a32;
  TO* out;
  float bc, cc;
  long long stride;
  int ld;
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
template <typename TX, typename TO>
struct EpiUpdate {
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
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    const TX* xb = x + b * xstride;
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = ac * Cvt<TX>::to_f(xb[(long long)(r0 + j) * ldx + c]) + v[j];
    TO* ob = out + b * ostride;
    if (!final_out) {
      emit4(ob, ldo, r0, c, v, mode);
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

// Plain fp32 store of C.
struct EpiStore {
  float* out;
  long long stride;
  int ld;
  __device__ void operator()(int b, int r0, int c, float v[4], int mode) const {
    emit4(out + b * stride, ld, r0, c, v, mode);
  }
};

// ------------------------------------------------------- staging ----------
// Four 16-byte registers of one thread's share of a tile. Members are named
// and indexed only with compile-time constants so that they stay in VGPRs.
struct Stage4 {
  u32x4_t v0, v1, v2, v3;
};
template <int I>
__device__ __forceinline__ u32x4_t& sget(Stage4& r) {
  if constexpr (I == 0) return r.v0;
  else if constexpr (I == 1) return r.v1;
  else if constexpr (I == 2) return r.v2;
  else return r.v3;
}
template <int I>
__device__ __forceinline__ const u32x4_t& sget(const Stage4& r) {
  if constexpr (I == 0) return r.v0;
  else if constexpr (I == 1) return r.v1;
  else if constexpr (I == 2) return r.v2;
  else return r.v3;
}

// A-type tile (rows x K, K contiguous): 1024 chunks of 16 B, 4 per thread;
// thread t owns rows t / 8 + 32 i, chunk t % 8.
template <int I, typename T>
__device__ __forceinline__ void load_row1(Stage4& r, const T* base, int ld, int row0, int k0) {
  const int t = threadIdx.x;
  const int row = (t >> 3) + 32 * I, ch = t & 7;
  const char* p = reinterpret_cast<const char*>(base + (long long)(row0 + row) * ld + k0) + ch * 16;
  sget<I>(r) = ld16(p);
}
template <typename T>
__device__ __forceinline__ void load_rows(Stage4& r, const T* base, int ld, int row0, int k0) {
  load_row1<0>(r, base, ld, row0, k0);
  load_row1<1>(r, base, ld, row0, k0);
  load_row1<2>(r, base, ld, row0, k0);
  load_row1<3>(r, base, ld, row0, k0);
}
template <int I>
__device__ __forceinline__ void store_row1(char* lds, const Stage4& r) {
  const int t = threadIdx.x;
  const int row = (t >> 3) + 32 * I, ch = t & 7;
  st16(lds + row * G_ROWB + ch * 16, sget<I>(r));
}
__device__ __forceinline__ void store_rows(char* lds, const Stage4& r) {
  store_row1<0>(lds, r);
  store_row1<1>(lds, r);
  store_row1<2>(lds, r);
  store_row1<3>(lds, r);
}

// NN B tile: global [K rows][N cols] (N contiguous) -> LDS [N rows][K].
// bf16: 64 x 128 tile, thread block 4 (k) x 8 (n): kb = t % 16, nb = t / 16.
__device__ __forceinline__ void load_nn(Stage4& r, const bf16_t* base, int ld, int k0, int n0) {
  const int t = threadIdx.x, kb = t & 15, nb = t >> 4;
  const bf16_t* p = base + (long long)(k0 + 4 * kb) * ld + n0 + 8 * nb;
  r.v0 = ld16(p);
  r.v1 = ld16(p + ld);
  r.v2 = ld16(p + 2 * (long long)ld);
  r.v3 = ld16(p + 3 * (long long)ld);
}
template <int P>
__device__ __forceinline__ void store_nn_pair(char* lds, const Stage4& r, int kb, int nb) {
  // column 2P: low halves of word P of rows k..k+3; column 2P + 1: high halves
  const uint32_t v0 = u4c(r.v0, P), v1 = u4c(r.v1, P), v2 = u4c(r.v2, P), v3 = u4c(r.v3, P);
  const u32x2_t lo = {__builtin_amdgcn_perm(v1, v0, 0x05040100u), __builtin_amdgcn_perm(v3, v2, 0x05040100u)};
  const u32x2_t hi = {__builtin_amdgcn_perm(v1, v0, 0x07060302u), __builtin_amdgcn_perm(v3, v2, 0x07060302u)};
  *reinterpret_cast<u32x2_t*>(lds + (8 * nb + 2 * P) * G_ROWB + 8 * kb) = lo;
  *reinterpret_cast<u32x2_t*>(lds + (8 * nb + 2 * P + 1) * G_ROWB + 8 * kb) = hi;
}
__device__ __forceinline__ void store_nn(char* lds, const Stage4& r, bf16_t) {
  const int t = threadIdx.x, kb = t & 15, nb = t >> 4;
  store_nn_pair<0>(lds, r, kb, nb);
  store_nn_pair<1>(lds, r, kb, nb);
  store_nn_pair<2>(lds, r, kb, nb);
  store_nn_pair<3>(lds, r, kb, nb);
}
// fp32: 32 x 128 tile, thread block 4 (k) x 4 (n): kb = t % 8, nb = t / 8.
__device__ __forceinline__ void load_nn(Stage4& r, const float* base, int ld, int k0, int n0) {
  const int t = threadIdx.x, kb = t & 7, nb = t >> 3;
  const float* p = base + (long long)(k0 + 4 * kb) * ld + n0 + 4 * nb;
  r.v0 = ld16(p);
  r.v1 = ld16(p + ld);
  r.v2 = ld16(p + 2 * (long long)ld);
  r.v3 = ld16(p + 3 * (long long)ld);
}
template <int J>
__device__ __forceinline__ void store_nn_col(char* lds, const Stage4& r, int kb, int nb) {
  const u32x4_t w = {r.v0[J], r.v1[J], r.v2[J], r.v3[J]};
  st16(lds + (4 * nb + J) * G_ROWB + 16 * kb, w);
}
__device__ __forceinline__ void store_nn(char* lds, const Stage4& r, float) {
  const int t = threadIdx.x, kb = t & 7, nb = t >> 3;
  store_nn_col<0>(lds, r, kb, nb);
  store_nn_col<1>(lds, r, kb, nb);
  store_nn_col<2>(lds, r, kb, nb);
  store_nn_col<3>(lds, r, kb, nb);
}

// fp32 source -> bf16 LDS (the bf16 filter keeps its iterate in fp32 and
// rounds it when it becomes a product operand). A thread holds two 16-byte
// halves per row: lo = floats 0..3, hi = floats 4..7 of its 8-element chunk.
struct Stage8 {
  Stage4 lo, hi;
};
template <int I>
__device__ __forceinline__ void load_row1_f(Stage8& r, const float* base, int ld, int row0, int k0) {
  const int t = threadIdx.x;
  const int row = (t >> 3) + 32 * I, ch = t & 7;
  const float* p = base + (long long)(row0 + row) * ld + k0 + 8 * ch;
  sget<I>(r.lo) = ld16(p);
  sget<I>(r.hi) = ld16(p + 4);
}
__device__ __forceinline__ u32x4_t pack8(const u32x4_t& a, const u32x4_t& b) {
  return u32x4_t{pack_bf2(__uint_as_float(a[0]), __uint_as_float(a[1])),
                 pack_bf2(__uint_as_float(a[2]), __uint_as_float(a[3])),
                 pack_bf2(__uint_as_float(b[0]), __uint_as_float(b[1])),
                 pack_bf2(__uint_as_float(b[2]), __uint_as_float(b[3]))};
}
template <int I>
__device__ __forceinline__ void store_row1_f(char* lds, const Stage8& r) {
  const int t = threadIdx.x;
  const int row = (t >> 3) + 32 * I, ch = t & 7;
  st16(lds + row * G_ROWB + ch * 16, pack8(sget<I>(r.lo), sget<I>(r.hi)));
}
// NN, fp32 source: 64 (k) x 128 (n) tile, thread block 4 (k) x 8 (n).
template <int I>
__device__ __forceinline__ float nnf(const Stage8& r, int c) {
  return __uint_as_float(c < 4 ? sget<I>(r.lo)[c] : sget<I>(r.hi)[c - 4]);
}
template <int P>
__device__ __forceinline__ void store_nn_pair_f(char* lds, const Stage8& r, int kb, int nb) {
  const u32x2_t lo = {pack_bf2(nnf<0>(r, 2 * P), nnf<1>(r, 2 * P)), pack_bf2(nnf<2>(r, 2 * P), nnf<3>(r, 2 * P))};
  const u32x2_t hi = {pack_bf2(nnf<0>(r, 2 * P + 1), nnf<1>(r, 2 * P + 1)),
                      pack_bf2(nnf<2>(r, 2 * P + 1), nnf<3>(r, 2 * P + 1))};
  *reinterpret_cast<u32x2_t*>(lds + (8 * nb + 2 * P) * G_ROWB + 8 * kb) = lo;
  *reinterpret_cast<u32x2_t*>(lds + (8 * nb + 2 * P + 1) * G_ROWB + 8 * kb) = hi;
}

// Staging policy per (LDS/MFMA type T, source type S).
template <typename T, typename S> struct Stager;
template <typename T> struct Stager<T, T> {
  using Reg = Stage4;
  __device__ __forceinline__ static void rows(Reg& r, const T* b, int ld, int row0, int k0) {
    load_rows(r, b, ld, row0, k0);
  }
  __device__ __forceinline__ static void rows_st(char* lds, const Reg& r) { store_rows(lds, r); }
  __device__ __forceinline__ static void nn(Reg& r, const T* b, int ld, int k0, int n0) { load_nn(r, b, ld, k0, n0); }
  __device__ __forceinline__ static void nn_st(char* lds, const Reg& r) { store_nn(lds, r, T{}); }
};
template <> struct Stager<bf16_t, float> {
  using Reg = Stage8;
  __device__ __forceinline__ static void rows(Reg& r, const float* b, int ld, int row0, int k0) {
    load_row1_f<0>(r, b, ld, row0, k0);
    load_row1_f<1>(r, b, ld, row0, k0);
    load_row1_f<2>(r, b, ld, row0, k0);
    load_row1_f<3>(r, b, ld, row0, k0);
  }
  __device__ __forceinline__ static void rows_st(char* lds, const Reg& r) {
    store_row1_f<0>(lds, r);
    store_row1_f<1>(lds, r);
    store_row1_f<2>(lds, r);
    store_row1_f<3>(lds, r);
  }
  __device__ __forceinline__ static void nn(Reg& r, const float* b, int ld, int k0, int n0) {
    const int t = threadIdx.x, kb = t & 15, nb = t >> 4;
    const float* p = b + (long long)(k0 + 4 * kb) * ld + n0 + 8 * nb;
    r.lo.v0 = ld16(p);
    r.hi.v0 = ld16(p + 4);
    r.lo.v1 = ld16(p + ld);
    r.hi.v1 = ld16(p + ld + 4);
    r.lo.v2 = ld16(p + 2 * (long long)ld);
    r.hi.v2 = ld16(p + 2 * (long long)ld + 4);
    r.lo.v3 = ld16(p + 3 * (long long)ld);
    r.hi.v3 = ld16(p + 3 * (long long)ld + 4);
  }
  __device__ __forceinline__ static void nn_st(char* lds, const Reg& r) {
    const int t = threadIdx.x, kb = t & 15, nb = t >> 4;
    store_nn_pair_f<0>(lds, r, kb, nb);
    store_nn_pair_f<1>(lds, r, kb, nb);
    store_nn_pair_f<2>(lds, r, kb, nb);
    store_nn_pair_f<3>(lds, r, kb, nb);
  }
};

// ---------------------------------------------------------- compute -------
template <typename T>
__device__ __forceinline__ void tile_mma(const char* la, const char* lb, f32x16_t acc[2][2],
                                         int wm, int wn, int lane) {
  const int r32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    u32x4_t a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      a[i] = ld16(la + (wm * 64 + i * 32 + r32) * G_ROWB + (2 * g + h) * 16);
      b[i] = ld16(lb + (wn * 64 + i * 32 + r32) * G_ROWB + (2 * g + h) * 16);
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        if constexpr (sizeof(T) == 2) {
          acc[mi][ni] = mfma32_bf16(a[mi], b[ni], acc[mi][ni]);
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
template <typename T, typename SA, typename SB, bool B_NN, bool SYM, typename Epi>
__global__ __launch_bounds__(G_THREADS, 2) void gemm_kernel(const SA* __restrict__ A,
                                                            const SB* __restrict__ B,
                                                            GemmShape sh, Epi epi) {
  using StA = Stager<T, SA>;
  using StB = Stager<T, SB>;
  constexpr int BK = GemmK<T>::BK;
  __shared__ __attribute__((aligned(16))) char lds[4 * G_TILEB];
  const int tiles_m = sh.M / G_BM, tiles_n = sh.N / G_BN;
  const int per = SYM ? tiles_m * (tiles_m + 1) / 2 : tiles_m * tiles_n;
  const int lid = xcd_remap(blockIdx.x, per * sh.batch);
  const int b = lid / per;
  int t = lid - b * per, tm, tn;
  if (SYM) {
    sym_tile(t, tiles_m, tm, tn);
  } else {
    tm = t / tiles_n;
    tn = t - tm * tiles_n;
  }
  const int m0 = tm * G_BM, n0 = tn * G_BN;
  const SA* Ab = A + b * sh.sa;
  const SB* Bb = B + b * sh.sb;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int wm = wave >> 1, wn = wave & 1;

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  typename StA::Reg ra;
  typename StB::Reg rb;
  const int nk = sh.K / BK;
  StA::rows(ra, Ab, sh.lda, m0, 0);
  if constexpr (B_NN) StB::nn(rb, Bb, sh.ldb, 0, n0);
  else StB::rows(rb, Bb, sh.ldb, n0, 0);
  StA::rows_st(lds, ra);
  if constexpr (B_NN) StB::nn_st(lds + G_TILEB, rb);
  else StB::rows_st(lds + G_TILEB, rb);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int k0 = (kt + 1) * BK;
      StA::rows(ra, Ab, sh.lda, m0, k0);
      if constexpr (B_NN) StB::nn(rb, Bb, sh.ldb, k0, n0);
      else StB::rows(rb, Bb, sh.ldb, n0, k0);
    }
    tile_mma<T>(lds + cur * 2 * G_TILEB, lds + cur * 2 * G_TILEB + G_TILEB, acc, wm, wn, lane);
    if (more) {
      char* nxt = lds + (cur ^ 1) * 2 * G_TILEB;
      StA::rows_st(nxt, ra);
      if constexpr (B_NN) StB::nn_st(nxt + G_TILEB, rb);
      else StB::rows_st(nxt + G_TILEB, rb);
    }
    __syncthreads();
  }

  const int mode = SYM ? (tm == tn ? EMIT_SYM_DIAG : EMIT_SYM_OFF) : EMIT_FULL;
  const int r32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v[4] = {acc[mi][ni][4 * i], acc[mi][ni][4 * i + 1], acc[mi][ni][4 * i + 2],
                      acc[mi][ni][4 * i + 3]};
        const int r0 = m0 + wm * 64 + mi * 32 + 8 * i + 4 * h;
        const int c = n0 + wn * 64 + ni * 32 + r32;
        epi(b, r0, c, v, mode);
      }
}

// Host launcher (errors surface through hipGetLastError at the end of a call).
template <typename T, bool B_NN, bool SYM, typename SA, typename SB, typename Epi>
void launch_gemm(const SA* A, const SB* B, const GemmShape& sh, const Epi& epi, hipStream_t stream) {
  const int tm = sh.M / G_BM, tn = sh.N / G_BN;
  const long long per = SYM ? (long long)tm * (tm + 1) / 2 : (long long)tm * tn;
  const long long blocks = per * sh.batch;
  if (blocks <= 0) return;
  hipLaunchKernelGGL((gemm_kernel<T, SA, SB, B_NN, SYM, Epi>), dim3((unsigned)blocks), dim3(G_THREADS), 0,
                     stream, A, B, sh, epi);
}

}  // namespace sd
