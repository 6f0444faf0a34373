// Tall-skinny products of the randomized SVD and the subspace step, the
// Gaussian sketch, and the canonical padded copy of an input batch.
//
// Panels are stored transposed: a (len x c) panel P lives as Pt[c][ld] with
// each column contiguous, zero beyond len.
//
//   ts_xtw:  Pt[j][n] = sum_i W[i][j] X[i][n]   (P = X^T W; X is s x l)
//   ts_xw:   Pt[j][i] = sum_n W[n][j] X[i][n]   (P = X W)
//
// Both stream X once and are bound by HBM; MFMA 16 x 16 blocks carry the
// products (bf16 operands with fp32 accumulation, or fp32). W is fp32 and is
// rounded to bf16 when it feeds a bf16 product. ACC64 (fp32 X only): the
// products run on the fp64 MFMA (v_mfma_f64_16x16x4f64) and accumulate in
// fp64; the results are rounded to fp32 once. Its operands sit in the lanes
// as the fp32 16 x 16 x 4 form's (A[i][k] in lane i + 16 k, B[k][j] in lane
// j + 16 k), but result item r of lane l is row 4 r + l / 16 of column
// l % 16, where the fp32 form has row 4 (l / 16) + r (checked on the GPU
// with an in-bounds probe over one block).
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace sd {

// 8 consecutive fp32 values -> 8 bf16 in 16 bytes.
__device__ __forceinline__ u32x4_t f8_to_bf8(const float* p) {
  const f32x4_t a = *reinterpret_cast<const f32x4_t*>(p);
  const f32x4_t b = *reinterpret_cast<const f32x4_t*>(p + 4);
  return u32x4_t{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(b[0], b[1]), pack_bf2(b[2], b[3])};
}

typedef double f64x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f64x4_t mfma16_f64(double a, double b, f64x4_t c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
// Accumulator of the fp32 skinny products: four fp32 or fp64 values.
template <bool ACC64>
struct SkAcc {
  typedef f32x4_t V;
  __device__ __forceinline__ static V mma(float a, float b, V c) { return mfma16_f32(a, b, c); }
  __device__ __forceinline__ static float get(const V& v, int j) { return v[j]; }
  // row of result item r in lane group q = lane / 16
  __device__ __forceinline__ static int row(int q, int r) { return 4 * q + r; }
};
template <>
struct SkAcc<true> {
  typedef f64x4_t V;
  __device__ __forceinline__ static V mma(float a, float b, V c) { return mfma16_f64((double)a, (double)b, c); }
  __device__ __forceinline__ static float get(const V& v, int j) { return (float)v[j]; }
  __device__ __forceinline__ static int row(int q, int r) { return 4 * r + q; }
};

// ------------------------------------------------------------ X^T W -------
// Grid: (l_pad / 128) * batch work-groups of 256 threads. MJ = ceil(rp / 16).
template <typename T, int MJ, bool ACC64 = false>
__global__ __launch_bounds__(256) void ts_xtw_kernel(const T* __restrict__ X, long long sx, int ldx,
                                                     int s_pad, int l_pad, const float* __restrict__ Wt,
                                                     long long sw, int ldw, int rp, float* __restrict__ Pt,
                                                     long long sp, int ldp, int batch) {
  constexpr int BK = GemmK<T>::BK;
  __shared__ __attribute__((aligned(16))) char lds[2 * G_TILEB];
  const int nslab = l_pad / 128;
  const int lid = xcd_remap(blockIdx.x, nslab * batch);
  const int b = lid / nslab, n0 = (lid - b * nslab) * 128;
  const T* Xb = X + b * sx;
  const float* Wb = Wt + b * sw;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int r16 = lane & 15, q = lane >> 4;
  static_assert(!ACC64 || sizeof(T) == 4, "fp64 accumulation serves the fp32 products");
  using Acc = SkAcc<ACC64>;

  typename Acc::V acc[MJ][2];
#pragma unroll
  for (int m = 0; m < MJ; ++m) acc[m][0] = acc[m][1] = typename Acc::V{};

  NNStager<128, 256, T, T> rb;
  const int nk = s_pad / BK;
  rb.load(Xb, ldx, 0, n0);
  rb.store(lds);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const int i0 = kt * BK;
    const bool more = kt + 1 < nk;
    if (more) rb.load(Xb, ldx, i0 + BK, n0);
    const char* ls = lds + cur * G_TILEB;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4_t bfr[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) bfr[nb] = ld16(ls + ((2 * wave + nb) * 16 + r16) * G_ROWB + (4 * u + q) * 16);
#pragma unroll
      for (int m = 0; m < MJ; ++m) {
        const int j = m * 16 + r16;
        if constexpr (sizeof(T) == 2) {
          u32x4_t a = {0u, 0u, 0u, 0u};
          if (j < rp) a = f8_to_bf8(Wb + (long long)j * ldw + i0 + 32 * u + 8 * q);
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            if constexpr (!ACC64) acc[m][nb] = mfma16_bf16(a, bfr[nb], acc[m][nb]);
          }
        } else {
          f32x4_t af = {0.f, 0.f, 0.f, 0.f};
          if (j < rp) af = *reinterpret_cast<const f32x4_t*>(Wb + (long long)j * ldw + i0 + 16 * u + 4 * q);
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][nb] = Acc::mma(af[t], u4f(bfr[nb], t), acc[m][nb]);
          }
        }
      }
    }
    if (more) rb.store(lds + (cur ^ 1) * G_TILEB);
    __syncthreads();
  }
  float* Pb = Pt + b * sp;
#pragma unroll
  for (int m = 0; m < MJ; ++m)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int j = m * 16 + Acc::row(q, jj);
        if (j < rp) Pb[(long long)j * ldp + n0 + (2 * wave + nb) * 16 + r16] = Acc::get(acc[m][nb], jj);
      }
}

// -------------------------------------------------------------- X W -------
// Grid: (s_pad / 16) * batch work-groups; the 4 waves split K = l_pad and
// their partial sums are added in wave order.
template <typename T, int MJ, bool ACC64 = false>
__global__ __launch_bounds__(256) void ts_xw_kernel(const T* __restrict__ X, long long sx, int ldx,
                                                    int s_pad, int l_pad, const float* __restrict__ Wt,
                                                    long long sw, int ldw, int rp, float* __restrict__ Pt,
                                                    long long sp, int ldp, int batch) {
  static_assert(!ACC64 || sizeof(T) == 4, "fp64 accumulation serves the fp32 products");
  using Acc = SkAcc<ACC64>;
  __shared__ typename Acc::V red[4][MJ][WAVE];
  const int nrb = s_pad / 16;
  const int lid = xcd_remap(blockIdx.x, nrb * batch);
  const int b = lid / nrb, i0 = (lid - b * nrb) * 16;
  const T* Xb = X + b * sx;
  const float* Wb = Wt + b * sw;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int r16 = lane & 15, q = lane >> 4;
  const int klen = l_pad / 4, kbeg = wave * klen, kend = kbeg + klen;

  typename Acc::V acc[MJ];
#pragma unroll
  for (int m = 0; m < MJ; ++m) acc[m] = typename Acc::V{};

  const T* xrow = Xb + (long long)(i0 + r16) * ldx;
  if constexpr (sizeof(T) == 2) {
    for (int k = kbeg; k < kend; k += 32) {
      const u32x4_t bx = ld16(xrow + k + 8 * q);
#pragma unroll
      for (int m = 0; m < MJ; ++m) {
        const int j = m * 16 + r16;
        u32x4_t a = {0u, 0u, 0u, 0u};
        if (j < rp) a = f8_to_bf8(Wb + (long long)j * ldw + k + 8 * q);
        if constexpr (!ACC64) acc[m] = mfma16_bf16(a, bx, acc[m]);
      }
    }
  } else {
    for (int k = kbeg; k < kend; k += 16) {
      const f32x4_t bf = *reinterpret_cast<const f32x4_t*>(xrow + k + 4 * q);
#pragma unroll
      for (int m = 0; m < MJ; ++m) {
        const int j = m * 16 + r16;
        f32x4_t af = {0.f, 0.f, 0.f, 0.f};
        if (j < rp) af = *reinterpret_cast<const f32x4_t*>(Wb + (long long)j * ldw + k + 4 * q);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[m] = Acc::mma(af[t], bf[t], acc[m]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < MJ; ++m) red[wave][m][lane] = acc[m];
  __syncthreads();
  if (wave == 0) {
    float* Pb = Pt + b * sp;
#pragma unroll
    for (int m = 0; m < MJ; ++m) {
      typename Acc::V s = red[0][m][lane];
      s += red[1][m][lane];
      s += red[2][m][lane];
      s += red[3][m][lane];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int j = m * 16 + Acc::row(q, jj);
        if (j < rp) Pb[(long long)j * ldp + i0 + r16] = Acc::get(s, jj);
      }
    }
  }
}

// ------------------------------------------------------- Gaussian sketch --
// Philox4x32-10 (Salmon et al., SC 2011) and Box-Muller (in float64, then
// rounded to float32). Counter (call, matrix, stream, 0), key (seed lo, hi).
struct Philox {
  __host__ __device__ __forceinline__ static void round(uint32_t c[4], uint32_t k0, uint32_t k1) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
  __host__ __device__ static void gen(uint32_t out[4], uint32_t call, uint32_t matrix, uint32_t stream,
                             uint64_t seed) {
    uint32_t c[4] = {call, matrix, stream, 0u};
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int r = 0; r < 10; ++r) {
      round(c, k0, k1);
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    out[0] = c[0];
    out[1] = c[1];
    out[2] = c[2];
    out[3] = c[3];
  }
  // Four standard normals from one counter value.
  __host__ __device__ static void normals(float z[4], uint32_t call, uint32_t matrix, uint32_t stream,
                                 uint64_t seed) {
    uint32_t w[4];
    gen(w, call, matrix, stream, seed);
    const double scale = 5.9604644775390625e-08;   // 2^-24
    const double two_pi = 2.0 * 3.141592653589793;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const double u1 = ((double)(w[2 * p] >> 8) + 1.0) * scale;
      const double u2 = (double)(w[2 * p + 1] >> 8) * scale;
      const double rad = sqrt(-2.0 * log(u1));
      const double ang = two_pi * u2;
      z[2 * p] = (float)(rad * cos(ang));
      z[2 * p + 1] = (float)(rad * sin(ang));
    }
  }
};

// Split bf16 copy of a panel value: hi = bf16(v) and lo = bf16(v - hi)
// (v - hi is exact in fp32).
__device__ __forceinline__ void split_bf16(float v, bf16_t& hi, bf16_t& lo) {
  hi = f2bf(v);
  lo = f2bf(v - bf2f(hi));
}

// Omega^T as a [rows][ld] panel for every matrix: entry (i, j) of the s x rp
// sketch is Gaussian number j * s + i of stream 1 (four per Philox call);
// every other entry of the panel (rows rp .. rows - 1, columns s .. ld - 1)
// is written as zero. With Wt16, also the split bf16 copy [rows16][ld]
// (stride sw16): hi in row j, lo in row rp + j, zero rows 2 rp .. rows16 - 1.
// One thread per four consecutive columns of a row of either panel.
static __global__ void sketch_kernel(float* __restrict__ Wt, long long sw, int ld, int s, int rp, int rows,
                                     uint64_t seed, int batch, bf16_t* __restrict__ Wt16, long long sw16,
                                     int rows16) {
  const int quads = (ld + 3) / 4;
  const int nrow = Wt16 && rows16 > rows ? rows16 : rows;
  const long long per = (long long)nrow * quads;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= per * batch) return;
  const int b = (int)(gid / per);
  const int rem = (int)(gid - (long long)b * per);
  const int j = rem / quads, i0 = 4 * (rem - j * quads);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (j < rp && i0 < s) {
    const long long g0 = (long long)j * s + i0;
    const uint32_t c0 = (uint32_t)(g0 >> 2);
    const int off = (int)(g0 & 3), nv = s - i0 < 4 ? s - i0 : 4;
    float z[8];
    Philox::normals(z, c0, (uint32_t)b, 1u, seed);
    if (off + nv > 4) Philox::normals(z + 4, c0 + 1, (uint32_t)b, 1u, seed);
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (t < nv) v[t] = z[off + t];
  }
  const long long o = b * sw + (long long)j * ld + i0;
  const long long o16 = b * sw16 + (long long)j * ld + i0;
#pragma unroll
  for (int t = 0; t < 4; ++t)
    if (i0 + t < ld) {
      if (j < rows) Wt[o + t] = v[t];
      if (Wt16) {
        if (j < rp) {
          bf16_t hi, lo;
          split_bf16(v[t], hi, lo);
          Wt16[o16 + t] = hi;
          Wt16[o16 + (long long)rp * ld + t] = lo;
        } else if (j >= 2 * rp && j < rows16) {
          Wt16[o16 + t] = 0;
        }
      }
    }
}

// A caller-supplied sketch [batch][rp][s] as the same zero-padded panels.
static __global__ void sketch_copy_kernel(float* __restrict__ Wt, long long sw, int ld, const float* __restrict__ src,
                                          int s, int rp, int rows, int batch, bf16_t* __restrict__ Wt16,
                                          long long sw16, int rows16) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int nrow = Wt16 && rows16 > rows ? rows16 : rows;
  const long long per = (long long)nrow * ld;
  if (gid >= per * batch) return;
  const int b = (int)(gid / per);
  const long long r = gid - (long long)b * per;
  const int j = (int)(r / ld), i = (int)(r - (long long)j * ld);
  const float v = (j < rp && i < s) ? src[((long long)b * rp + j) * s + i] : 0.f;
  if (j < rows) Wt[b * sw + r] = v;
  if (Wt16) {
    if (j < rp) {
      bf16_t hi, lo;
      split_bf16(v, hi, lo);
      Wt16[b * sw16 + r] = hi;
      Wt16[b * sw16 + r + (long long)rp * ld] = lo;
    } else if (j >= 2 * rp && j < rows16) {
      Wt16[b * sw16 + r] = 0;
    }
  }
}

// ----------------------------------------------------- canonical copy ----
// dst[b][i][n] (padded rows_pad x ld, zero outside rows x cols) from
// src[b] of shape rows x cols (row-major) or, with transpose, cols x rows.
template <typename T>
__global__ __launch_bounds__(256) void canon_copy_kernel(T* __restrict__ dst, long long sd_, int ldd, int rows_pad,
                                                         int cols_pad, const T* __restrict__ src, long long ss,
                                                         int rows, int cols, int transpose, int batch) {
  __shared__ T tile[32][33];
  const int tr = rows_pad / 32, tc = cols_pad / 32;
  const int per = tr * tc;
  const int b = blockIdx.x / per;
  if (b >= batch) return;
  const int t = blockIdx.x - b * per;
  const int r0 = (t / tc) * 32, c0 = (t % tc) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  const T* sb = src + b * ss;
  T* db = dst + b * sd_;
  if (!transpose) {
    for (int y = ty; y < 32; y += 8) {
      const int r = r0 + y, c = c0 + tx;
      T v = T(0);
      if (r < rows && c < cols) v = sb[(long long)r * cols + c];
      db[(long long)r * ldd + c] = v;
    }
  } else {
    // dst(r, c) = src(c, r); src is cols x rows.
    for (int y = ty; y < 32; y += 8) {
      const int sr = c0 + y, sc = r0 + tx;
      T v = T(0);
      if (sr < cols && sc < rows) v = sb[(long long)sr * rows + sc];
      tile[y][tx] = v;
    }
    __syncthreads();
    for (int y = ty; y < 32; y += 8) db[(long long)(r0 + y) * ldd + c0 + tx] = tile[tx][y];
  }
}

}  // namespace sd
