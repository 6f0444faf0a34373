// Element-wise passes with a low-rank term, streamed once through HBM:
//
//   out[i][n] = alpha * x[i][n] + sum_{j < kk} L[j][i] c[j] Rr[j][n]
//
// over a padded rows x cols domain (multiples of 128). Used for the residual
// norm of the deflated polar factor (sum of out^2 per tile, no output), the
// padded start X0 of Alg. 1 and Alg. 2 and the PSD residual R of Alg. 2.
// Per-matrix alpha, c and kk are read from device memory so that gate
// decisions never leave the GPU.
//
// The float32 Muon start takes the two-term form (ACC64)
//
//   out[i][n] = alpha * (x[i][n] + sum_j L[j][i] c[j] Rr[j][n]) + sum_j L[j][i] c2[j] Rr[j][n]
//
// with the first sum and the difference in float64: the float32 factors'
// products are exact there, so R = x - V S U^T is formed to float32 rounding
// of R itself instead of the head's (a head s_1 / nu times larger than R
// otherwise leaves 2^-24 s_1 / nu of rounding in R / nu, which the filter's
// slope at zero amplifies).
#pragma once

#include "common.hpp"

namespace sd {

struct LowRankArgs {
  const void* x;
  long long sx;
  int ldx;
  const float* L;     // [b][j][ld_l]
  long long sl;
  int ldl;
  const float* Rr;    // [b][j][ld_r]
  long long sr;
  int ldr;
  const float* coef;  // [b][kmax]
  const float* coef2; // [b][kmax], two-term form only (ACC64)
  const int* kk;      // [b] or null (then kconst)
  int kconst;
  const float* alpha; // [b] or null (then 1)
  void* out;          // null: no output
  long long so;
  int ldo;
  bf16_t* out16;      // optional bf16 copy of out (same layout)
  int8_t* out_lo;     // with out16: e4m3 residual byte of out against bf16(out) (state_pack8)
  f16_t* xs16;        // optional fp16(alpha * x) (same layout as out)
  float* sumsq;       // [b][tiles] or null
  int rows_pad, cols_pad, kmax, batch;
};

template <typename T>
__device__ __forceinline__ void store8(T* p, const float v[8]);
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* p, const float v[8]) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]),
                                            pack_bf2(v[4], v[5]), pack_bf2(v[6], v[7]));
}
template <>
__device__ __forceinline__ void store8<float>(float* p, const float v[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// Eight consecutive elements as loaded (raw bits), converted after the wait.
template <typename T>
struct Raw8;
template <>
struct Raw8<bf16_t> {
  uint4 u;
  __device__ __forceinline__ void load(const bf16_t* p) { u = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void get(float v[8]) const {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ void get(float v[8]) const {
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
};

// 128 x 128 tile per work-group; thread t owns rows 8 (t / 16) .. +7 and
// columns 8 (t % 16) .. +7. WPE: minimum waves per SIMD the register
// allocation must allow (4 for the bf16 passes of the Muon start, which
// would otherwise take 130 registers and three waves: the passes are bound
// by the X loads in flight, and a fourth work-group per CU adds a third).
template <typename TX, typename TO, int KM, int WPE = 1, bool ACC64 = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE))) void lowrank_kernel(LowRankArgs a) {
  __shared__ __attribute__((aligned(16))) float ls[KM][128];
  __shared__ __attribute__((aligned(16))) float rs[KM][128];
  __shared__ __attribute__((aligned(16))) float l2s[ACC64 ? KM : 1][128];
  __shared__ float cs[ACC64 ? KM : 1];
  __shared__ float red[4];
  const int tr = a.rows_pad / 128, tc = a.cols_pad / 128, per = tr * tc;
  const int lid = xcd_remap(blockIdx.x, per * a.batch);
  const int b = lid / per, t = lid - b * per;
  const int i0 = (t / tc) * 128, n0 = (t % tc) * 128;
  const int tid = threadIdx.x;
  const int rg = tid >> 4, cg = tid & 15;
  // Every load is issued before any of them is used: the low-rank panels
  // and their coefficients (all kmax rows: the coefficients past the
  // per-matrix count are zero, so no load waits on that count; rows past
  // kmax load row kmax - 1 and are not stored), then the thread's X values,
  // whose latency overlaps the low-rank product. (Scaling a panel value as
  // it arrives made every panel load wait for the one before.)
  constexpr int PER = KM * 128 / 256;
  float lv[PER], cv[PER], rv[PER], c2v[ACC64 ? PER : 1];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = tid + 256 * u, j = e >> 7, x = e & 127;
    const int jc = j < a.kmax ? j : a.kmax - 1;
    lv[u] = a.L[b * a.sl + (long long)jc * a.ldl + i0 + x];
    cv[u] = a.coef[b * a.kmax + jc];
    rv[u] = a.Rr[b * a.sr + (long long)jc * a.ldr + n0 + x];
    if constexpr (ACC64) c2v[u] = a.coef2 ? a.coef2[b * a.kmax + jc] : 0.f;
  }
  const TX* xb = reinterpret_cast<const TX*>(a.x) + b * a.sx;
  Raw8<TX> xr[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) xr[r].load(xb + (long long)(i0 + rg * 8 + r) * a.ldx + n0 + cg * 8);
  const int kk = a.kk ? a.kk[b] : a.kconst;
  const float alpha = a.alpha ? a.alpha[b] : 1.f;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = tid + 256 * u, j = e >> 7, x = e & 127;
    if (j < a.kmax) {
      if constexpr (ACC64) {
        ls[j][x] = lv[u];            // unscaled: the coefficient is applied in float64
        l2s[j][x] = lv[u] * c2v[u];
        if (x == 0) cs[j] = cv[u];
      } else {
        ls[j][x] = lv[u] * cv[u];
      }
      rs[j][x] = rv[u];
    }
  }
  __syncthreads();
  if constexpr (ACC64) {
    // two-term float32 start: R = x + sum_j L c R^T in float64, then
    // out = alpha R + sum_j L c2 R^T
    double accd[8][8];
    float acc2[8][8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        accd[r][c] = 0.0;
        acc2[r][c] = 0.f;
      }
    for (int j = 0; j < kk; ++j) {
      const double cj = (double)cs[j];
      double ld[8];
      float l2[8], rv8[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        ld[r] = (double)ls[j][rg * 8 + r] * cj;
        l2[r] = l2s[j][rg * 8 + r];
        rv8[r] = rs[j][cg * 8 + r];
      }
#pragma unroll
      for (int r = 0; r < 8; ++r)
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          accd[r][c] = fma(ld[r], (double)rv8[c], accd[r][c]);
          acc2[r][c] = fmaf(l2[r], rv8[c], acc2[r][c]);
        }
    }
    TO* ob = a.out ? reinterpret_cast<TO*>(a.out) + b * a.so : nullptr;
    double ssd = 0.0;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int i = i0 + rg * 8 + r;
      float v[8];
      xr[r].get(v);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const double rr = (double)v[c] + accd[r][c];
        ssd = fma(rr, rr, ssd);
        v[c] = (float)((double)alpha * rr) + acc2[r][c];
      }
      if (ob) store8<TO>(ob + (long long)i * a.ldo + n0 + cg * 8, v);
    }
    if (a.sumsq) {
      const float ss = (float)ssd;
      const float tot = block_sum(ss, red);
      if (tid == 0) a.sumsq[(long long)b * per + t] = tot;
    }
    return;
  }
  float acc[8][8];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[r][c] = 0.f;
  for (int j = 0; j < kk; ++j) {
    const float4 l0 = *reinterpret_cast<const float4*>(&ls[j][rg * 8]);
    const float4 l1 = *reinterpret_cast<const float4*>(&ls[j][rg * 8 + 4]);
    const float4 r0 = *reinterpret_cast<const float4*>(&rs[j][cg * 8]);
    const float4 r1 = *reinterpret_cast<const float4*>(&rs[j][cg * 8 + 4]);
    const float lv[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
    const float rv[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[r][c] = fmaf(lv[r], rv[c], acc[r][c]);
  }
  TO* ob = a.out ? reinterpret_cast<TO*>(a.out) + b * a.so : nullptr;
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int i = i0 + rg * 8 + r;
    float v[8];
    xr[r].get(v);
    if (a.xs16) {
      const long long o = b * a.so + (long long)i * a.ldo + n0 + cg * 8;
      *reinterpret_cast<u32x4_t*>(a.xs16 + o) =
          u32x4_t{pack_h2(alpha * v[0], alpha * v[1]), pack_h2(alpha * v[2], alpha * v[3]),
                  pack_h2(alpha * v[4], alpha * v[5]), pack_h2(alpha * v[6], alpha * v[7])};
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      v[c] = fmaf(alpha, v[c], acc[r][c]);
      ss = fmaf(v[c], v[c], ss);
    }
    if (ob) store8<TO>(ob + (long long)i * a.ldo + n0 + cg * 8, v);
    if (a.out16) {
      uint32_t nh[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) nh[q] = pack_bf2(v[2 * q], v[2 * q + 1]);
      const long long o = b * a.so + (long long)i * a.ldo + n0 + cg * 8;
      st16_nt(a.out16 + o, u32x4_t{nh[0], nh[1], nh[2], nh[3]});
      if (a.out_lo) st8_nt(a.out_lo + o, state_pack8(v, nh));
    }
  }
  if (a.sumsq) {
    ss = block_sum(ss, red);
    if (tid == 0) a.sumsq[(long long)b * per + t] = ss;
  }
}

// nu = sqrt(sum of the residual tiles) (float64: per-lane strided partial
// sums, then lane 0's butterfly total); alpha = 1/nu (0 for nu = 0) and the
// start coefficients c_j = -(s_j / nu - 1 / gamma) of
//   X0 = alpha X + sum_j L_j c_j R_j^T  =  R / nu + gamma^-1 L R^T
// (1 / gamma = 0 for the explicit restore). With coef_one, also the restore
// coefficients: 1 for the deflated components, 0 past them. With coef_g, the
// head coefficients of the two-term start (ACC64 lowrank_kernel): 1 / gamma
// for the deflated components. One wave per matrix.
// Residual floor: with k_eff > 0, a residual with nu <= rho ||X||_F, where
// ||X||_F^2 = sum_{j < k_eff} s_j^2 + nu^2 (U_k S_k V_k^T is the projection
// of X on the head), is rounding of the head's arithmetic: its components
// along the head directions are then not small against nu, and R / nu next
// to the padded head can leave the filter's convergence interval. Such a
// residual is dropped (alpha = 0: X0 = gamma^-1 L R^T, or 0 for the explicit
// restore) and flag 4 is raised in status.
static __global__ __launch_bounds__(64) void muon_finalize_kernel(const float* sumsq, int tiles, const float* sv,
                                                                  const int* keff, int kmax, float inv_gamma,
                                                                  float rho, float* alpha, float* coef_b,
                                                                  float* nu_dev, float* nu_user, float* coef_one,
                                                                  float* coef_g, int* status, int batch) {
  const int b = blockIdx.x, lane = threadIdx.x;
  double acc = 0.0;
  for (int t = lane; t < tiles; t += WAVE) acc += (double)sumsq[(long long)b * tiles + t];
  acc = wave_sum(acc);
  acc = __shfl(acc, 0, WAVE);
  const double nu = sqrt(acc);
  const int ke = keff ? keff[b] : 0;
  double head = 0.0;
  for (int j = 0; j < ke; ++j) head += (double)sv[b * kmax + j] * (double)sv[b * kmax + j];
  const bool floored = ke > 0 && nu <= (double)rho * sqrt(head + acc);
  const double inv = (nu > 0.0 && !floored) ? 1.0 / nu : 0.0;
  if (lane == 0) {
    alpha[b] = (float)inv;
    nu_dev[b] = (float)nu;
    if (nu_user) nu_user[b] = (float)nu;
    if (floored && status) atomicOr(status, 4);
  }
  for (int j = lane; j < kmax; j += WAVE) {
    coef_b[b * kmax + j] = j < ke ? (float)(-((double)sv[b * kmax + j] * inv - (double)inv_gamma)) : 0.f;
    if (coef_one) coef_one[b * kmax + j] = j < ke ? 1.f : 0.f;
    if (coef_g) coef_g[b * kmax + j] = j < ke ? inv_gamma : 0.f;
  }
}

static __global__ void fill_kernel(float* p, long long n, float v) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}
static __global__ void fill_int_kernel(int* p, long long n, int v) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Padded canonical iterate -> caller layout (rows x cols, or its transpose).
template <typename TX, typename TO>
__global__ void store_out_kernel(const TX* x, long long sx, int ldx, TO* out, long long so, int rows, int cols,
                                 int transpose, int batch) {
  const long long per = (long long)rows * cols;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= per * batch) return;
  const int b = (int)(gid / per);
  const long long r = gid - (long long)b * per;
  if (!transpose) {
    const int i = (int)(r / cols), n = (int)(r - (long long)i * cols);
    out[b * so + r] = Cvt<TO>::from_f(Cvt<TX>::to_f(x[b * sx + (long long)i * ldx + n]));
  } else {
    // out is cols x rows: out[n][i] = x[i][n]
    const int n = (int)(r / rows), i = (int)(r - (long long)n * rows);
    out[b * so + r] = Cvt<TO>::from_f(Cvt<TX>::to_f(x[b * sx + (long long)i * ldx + n]));
  }
}

// Panel (c x ld, transposed storage) -> caller matrix (len x c, row-major).
static __global__ void panel_to_rows_kernel(const float* pt, int ld, int c, int len, float* out) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)len * c) return;
  const int x = (int)(gid / c), j = (int)(gid - (long long)x * c);
  out[gid] = pt[(long long)j * ld + x];
}

// Caller matrix (len x c, row-major) -> panel (c x ld), zero beyond len.
static __global__ void rows_to_panel_kernel(const float* in, int c, int len, int ld, float* pt) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)c * ld) return;
  const int j = (int)(gid / ld), x = (int)(gid - (long long)j * ld);
  pt[gid] = x < len ? in[(long long)x * c + j] : 0.f;
}

// PSD output (Alg. 2 restore and symmetrization): with C = R g(X0) and the
// restored head H = sum_{p < kk} cp[p] u_p u_p^T, P_raw = R / 2 + C / 2 + H and
//   P = (P_raw + P_raw^T) / 2 = (R + R^T) / 4 + (C + C^T) / 4 + H.
// Every term is evaluated so that P[i][j] and P[j][i] see the same operations
// on swapped operands (sums are commutative, H uses cp * (u_i u_j)), hence P
// is exactly symmetric. 64 x 64 tiles; the transposed tiles and the head's
// coefficients go through LDS (a coefficient read from global memory inside
// the head sum was re-read after every store, which may alias it).
template <int KM>
__global__ __launch_bounds__(256) void psd_out_kernel(const float* __restrict__ R, const float* __restrict__ C,
                                                      int ld, const float* __restrict__ Ut, int ldu,
                                                      const float* __restrict__ coef_p, const int* kk_dev, int n,
                                                      int n_pad, float* __restrict__ out) {
  __shared__ float ct[64][65];
  __shared__ float rt[64][65];
  __shared__ float ui[KM][64];
  __shared__ float uj[KM][64];
  __shared__ float cps[KM];
  const int tiles = n_pad / 64;
  const int i0 = (blockIdx.x / tiles) * 64, j0 = (blockIdx.x % tiles) * 64;
  const int tid = threadIdx.x;
  const int kk = kk_dev ? *kk_dev : 0;
  for (int e = tid; e < 64 * 64; e += 256) {
    const int r = e >> 6, c = e & 63;
    const long long src = (long long)(j0 + r) * ld + i0 + c;   // element (j0 + r, i0 + c)
    ct[c][r] = C[src];
    rt[c][r] = R[src];
  }
  for (int e = tid; e < kk * 64; e += 256) {
    const int p = e >> 6, x = e & 63;
    ui[p][x] = Ut[(long long)p * ldu + i0 + x];
    uj[p][x] = Ut[(long long)p * ldu + j0 + x];
  }
  if (tid < kk) cps[tid] = coef_p[tid];
  __syncthreads();
  const int tx = tid & 63, ty = tid >> 6;
  for (int r = ty; r < 64; r += 4) {
    const int i = i0 + r, j = j0 + tx;
    float h = 0.f;
    for (int p = 0; p < kk; ++p) h = fmaf(cps[p], ui[p][r] * uj[p][tx], h);
    const long long ij = (long long)i * ld + j;
    const float v = 0.25f * (R[ij] + rt[r][tx]) + 0.25f * (C[ij] + ct[r][tx]) + h;
    if (i < n && j < n) out[(long long)i * n + j] = v;
  }
}

}  // namespace sd
