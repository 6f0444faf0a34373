// Deflated PSD projection (Alg. 2) with the Lanczos scale of App. E.1: host
// orchestration, the Lanczos kernels and the C entry points.
//
//   (J - 1) x [Zt = Z V, CholQR]  ->  Zt = Z V  ->  Rayleigh-Ritz (float64)
//   R = Z - U_I diag(lam_I) U_I^T            (one streaming pass)
//   theta = Lanczos upper estimate of ||R||_2 (GEMVs with R, float64 recurrences)
//   X0 = R / theta + gamma^-1 U_I sign(lam_I) U_I^T
//   g = L steps of X <- a X + (b A + c A^2) X, A = X X (symmetric tiles only)
//   C = R g  ->  P = R / 2 + (C + C^T) / 4 + U_I max(lam_I, 0) U_I^T
//   Qwarm <- CholQR(Zt)
// With nothing deflated the same kernels run with R = Z, which is the
// baseline projection of eq:baseline_projection.
#include "host.hpp"
#include "wide.hpp"

namespace sd {

constexpr int LZ_MAX = 64;   // largest Lanczos step count
constexpr int PSD_NARROW_MAX = 32;   // widest tracked basis whose K x K problems stay in one work-group

// y[i] = sum_j A[i][j] x[j]; one wave per row, four rows per work-group.
__global__ __launch_bounds__(256) void gemv_kernel(const float* __restrict__ A, int ld, int n_pad,
                                                   const float* __restrict__ x, float* __restrict__ y) {
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  const int row = blockIdx.x * 4 + wave;
  if (row >= n_pad) return;
  const float* a = A + (long long)row * ld;
  float acc = 0.f;
  for (int c = lane * 4; c < n_pad; c += 4 * WAVE) {
    const float4 av = *reinterpret_cast<const float4*>(a + c);
    const float4 xv = *reinterpret_cast<const float4*>(x + c);
    acc = fmaf(av.x, xv.x, acc);
    acc = fmaf(av.y, xv.y, acc);
    acc = fmaf(av.z, xv.z, acc);
    acc = fmaf(av.w, xv.w, acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) y[row] = acc;
}

struct LanczosState {
  double alpha[LZ_MAX];
  double beta[LZ_MAX];
  int active;      // number of Lanczos vectors that may be used
  int steps;       // alpha entries computed
  double rho;
  double y[LZ_MAX];   // the largest Ritz vector of the tridiagonal matrix
};

// q_0 = g / ||g|| with g the Philox Gaussians of stream 2 (n entries, zero
// padding). One work-group of 1024 threads.
__global__ __launch_bounds__(1024) void lanczos_init_kernel(float* Q, int n, int n_pad, int m, uint64_t seed,
                                                            LanczosState* st) {
  __shared__ double red[16];
  const int tid = threadIdx.x;
  double ss = 0.0;
  for (int c = tid; 4 * c < n_pad; c += 1024) {
    float z[4];
    Philox::normals(z, (uint32_t)c, 0u, 2u, seed);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int i = 4 * c + t;
      const float v = i < n ? z[t] : 0.f;
      Q[i] = v;
      ss += (double)v * v;
    }
  }
  ss = block_sum(ss, red);
  const float inv = (float)(1.0 / sqrt(ss));
  for (int i = tid; i < n_pad; i += 1024) Q[i] = (float)((double)Q[i] / sqrt(ss));
  (void)inv;
  if (tid == 0) {
    st->active = m;
    st->steps = 0;
    st->rho = 0.0;
  }
}

// One Lanczos step on B = R^2 with w = B q_j already computed, on one
// work-group (n_pad below 8192: one launch instead of four):
//   alpha_j = q_j . w;  w -= alpha_j q_j + beta_{j-1} q_{j-1};
//   two classical Gram-Schmidt passes against q_0..q_j;
//   beta_j = ||w||; q_{j+1} = w / beta_j (a zero beta ends the run).
// Thread t keeps the float4 chunks t and t + 1024 of w in registers for the
// whole step; the basis vectors are read four at a time with every load of
// a batch issued before its first use (a loop that waited on each load made
// the step a chain of memory round trips), and a pass's products are
// reduced per wave, then over the waves, with one barrier.
constexpr int LS_CH = 2;   // float4 chunks per thread: n_pad / 4 <= 2048
constexpr int LS_B = 4;    // basis vectors per load batch
// p[i] when ok, else zeros; the load always reads an in-bounds element (p[0]
// when not ok) and the zeros are a value select, so the pointer stays a
// global one (selecting between a global element and a local zero made
// every load a flat one).
__device__ __forceinline__ float4 ld4_or0(const float4* __restrict__ p, long long i, bool ok) {
  const float4 v = p[ok ? i : 0];
  return ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
}
__device__ __forceinline__ float ld_or0(const float* __restrict__ p, long long i, bool ok) {
  const float v = p[ok ? i : 0];
  return ok ? v : 0.f;
}
__device__ __forceinline__ double dot4(const float4& a, const float4& b) {
  return (double)a.x * b.x + (double)a.y * b.y + (double)a.z * b.z + (double)a.w * b.w;
}
__global__ __launch_bounds__(1024) void lanczos_step_kernel(float* Q, int n_pad, float* w, int j, int m,
                                                            LanczosState* st) {
  __shared__ double red[16];
  __shared__ double part[LZ_MAX][1024 / WAVE];
  __shared__ double h[LZ_MAX];
  const int tid = threadIdx.x, wave = tid / WAVE, lane = tid & (WAVE - 1);
  if (j >= st->active) return;
  const int n4 = n_pad / 4;
  const float4* Q4 = reinterpret_cast<const float4*>(Q);
  float4* w4 = reinterpret_cast<float4*>(w);
  int idx[LS_CH];
  bool ok[LS_CH];
  float4 wr[LS_CH], qj[LS_CH], qp[LS_CH];
  const double bprev = j > 0 ? st->beta[j - 1] : 0.0;
#pragma unroll
  for (int c = 0; c < LS_CH; ++c) {
    idx[c] = tid + 1024 * c;
    ok[c] = idx[c] < n4;
    wr[c] = ld4_or0(w4, idx[c], ok[c]);
    qj[c] = ld4_or0(Q4, (long long)j * n4 + idx[c], ok[c]);
    qp[c] = ld4_or0(Q4, (long long)(j > 0 ? j - 1 : 0) * n4 + idx[c], ok[c] && j > 0);
  }
  double acc = 0.0;
#pragma unroll
  for (int c = 0; c < LS_CH; ++c) acc += dot4(qj[c], wr[c]);
  const double a = block_sum(acc, red);
#pragma unroll
  for (int c = 0; c < LS_CH; ++c) {
    wr[c].x = (float)((double)wr[c].x - a * qj[c].x - (j > 0 ? bprev * qp[c].x : 0.0));
    wr[c].y = (float)((double)wr[c].y - a * qj[c].y - (j > 0 ? bprev * qp[c].y : 0.0));
    wr[c].z = (float)((double)wr[c].z - a * qj[c].z - (j > 0 ? bprev * qp[c].z : 0.0));
    wr[c].w = (float)((double)wr[c].w - a * qj[c].w - (j > 0 ? bprev * qp[c].w : 0.0));
  }
  for (int pass = 0; pass < 2; ++pass) {
    for (int v0 = 0; v0 <= j; v0 += LS_B) {
      float4 qa[LS_B][LS_CH];
#pragma unroll
      for (int u = 0; u < LS_B; ++u)
#pragma unroll
        for (int c = 0; c < LS_CH; ++c)
          qa[u][c] = ld4_or0(Q4, (long long)(v0 + u) * n4 + idx[c], v0 + u <= j && ok[c]);
#pragma unroll
      for (int u = 0; u < LS_B; ++u) {
        if (v0 + u <= j) {   // uniform over the work-group
          double d = 0.0;
#pragma unroll
          for (int c = 0; c < LS_CH; ++c) d += dot4(qa[u][c], wr[c]);
          d = wave_sum(d);
          if (lane == 0) part[v0 + u][wave] = d;
        }
      }
    }
    __syncthreads();
    if (tid <= j) {
      double t = 0.0;
      for (int q = 0; q < 1024 / WAVE; ++q) t += part[tid][q];
      h[tid] = t;
    }
    __syncthreads();
    double t[LS_CH][4];
#pragma unroll
    for (int c = 0; c < LS_CH; ++c) {
      t[c][0] = wr[c].x;
      t[c][1] = wr[c].y;
      t[c][2] = wr[c].z;
      t[c][3] = wr[c].w;
    }
    for (int v0 = 0; v0 <= j; v0 += LS_B) {
      float4 qa[LS_B][LS_CH];
#pragma unroll
      for (int u = 0; u < LS_B; ++u)
#pragma unroll
        for (int c = 0; c < LS_CH; ++c)
          qa[u][c] = ld4_or0(Q4, (long long)(v0 + u) * n4 + idx[c], v0 + u <= j && ok[c]);
#pragma unroll
      for (int u = 0; u < LS_B; ++u) {
        if (v0 + u <= j) {
          const double hv = h[v0 + u];
#pragma unroll
          for (int c = 0; c < LS_CH; ++c) {
            t[c][0] -= hv * qa[u][c].x;
            t[c][1] -= hv * qa[u][c].y;
            t[c][2] -= hv * qa[u][c].z;
            t[c][3] -= hv * qa[u][c].w;
          }
        }
      }
    }
#pragma unroll
    for (int c = 0; c < LS_CH; ++c)
      wr[c] = make_float4((float)t[c][0], (float)t[c][1], (float)t[c][2], (float)t[c][3]);
    __syncthreads();   // part and h are reused by the next pass
  }
#pragma unroll
  for (int c = 0; c < LS_CH; ++c)
    if (ok[c]) w4[idx[c]] = wr[c];
  if (tid == 0) {
    st->alpha[j] = a;
    st->steps = j + 1;
  }
  if (j == m - 1) return;
  double nn = 0.0;
#pragma unroll
  for (int c = 0; c < LS_CH; ++c) nn += dot4(wr[c], wr[c]);
  const double beta = sqrt(block_sum(nn, red));
  if (beta == 0.0) {
    if (tid == 0) st->active = j + 1;
    return;
  }
  float4* qn = reinterpret_cast<float4*>(Q + (long long)(j + 1) * n_pad);
#pragma unroll
  for (int c = 0; c < LS_CH; ++c)
    if (ok[c])
      qn[idx[c]] = make_float4((float)((double)wr[c].x / beta), (float)((double)wr[c].y / beta),
                               (float)((double)wr[c].z / beta), (float)((double)wr[c].w / beta));
  if (tid == 0) st->beta[j] = beta;
}

// The same step spread over work-groups of 256 positions (one per thread),
// for n_pad from 8192 up (the one-work-group step grows with n: 187 us at
// n = 16384, against about 55 us here), in four launches:
//   dots:    h_v = q_v . w for v <= j (per-wave partial sums);
//   pass 1:  w -= sum_v h_v q_v, with alpha_j = h_j (this subtracts the
//            three-term recurrence's alpha_j q_j and beta_{j-1} q_{j-1} and
//            a first classical Gram-Schmidt pass in one), then the partial
//            products of the second pass;
//   pass 2:  w -= sum_v h'_v q_v, then the partial squares of w;
//   next:    beta_j = ||w||, q_{j+1} = w / beta_j (a zero beta ends the run).
// Every work-group reduces the partials itself (fixed order), so the steps
// need no atomics and are deterministic. A run that has ended (j >= active)
// returns at once.
constexpr int LZ_BLOCK = 256;
constexpr int LZ_MULTI_MIN = 8192;   // n_pad from which the step spreads over work-groups
static_assert(LZ_MULTI_MIN / 4 <= LS_CH * 1024, "the one-work-group step holds n_pad / 4 chunks in LS_CH per thread");

__host__ __device__ inline int lanczos_partials(int n_pad) { return 4 * ((n_pad + LZ_BLOCK - 1) / LZ_BLOCK); }

// h[v] (LDS) = sum over the partials of row v, v <= j; one wave per row.
__device__ __forceinline__ void lanczos_reduce(const double* part, int np4, int j, double* h) {
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  for (int v = wave; v <= j; v += LZ_BLOCK / WAVE) {
    double t = 0.0;
    for (int e = lane; e < np4; e += WAVE) t += part[(long long)v * np4 + e];
    t = wave_sum(t);
    if (lane == 0) h[v] = t;
  }
  __syncthreads();
}

// part[v][4 blk + wave] = sum over the wave's positions of q_v[i] y (v <= j).
__device__ __forceinline__ void lanczos_partial_dots(const float* Q, int n_pad, int j, int i, double y,
                                                     double* part, int np4) {
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
  for (int v0 = 0; v0 <= j; v0 += 8) {
    float q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = ld_or0(Q, (long long)(v0 + u) * n_pad + i, v0 + u <= j && i < n_pad);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (v0 + u <= j) {
        const double d = wave_sum((double)q[u] * y);
        if (lane == 0) part[(long long)(v0 + u) * np4 + 4 * blockIdx.x + wave] = d;
      }
    }
  }
}

__global__ __launch_bounds__(LZ_BLOCK) void lanczos_dots_kernel(const float* Q, int n_pad, const float* w, int j,
                                                                double* part, const LanczosState* st) {
  if (j >= st->active) return;
  const int i = blockIdx.x * LZ_BLOCK + threadIdx.x;
  const double y = (double)ld_or0(w, i, i < n_pad);
  lanczos_partial_dots(Q, n_pad, j, i, y, part, lanczos_partials(n_pad));
}

// pass 1 (last = 0): subtract, store alpha_j, partial dots of the result into
// out; pass 2 (last = 1): subtract, partial squares into out (row 0).
__global__ __launch_bounds__(LZ_BLOCK) void lanczos_pass_kernel(const float* Q, int n_pad, float* w, int j,
                                                                const double* in, double* out, int last,
                                                                LanczosState* st) {
  __shared__ double h[LZ_MAX];
  if (j >= st->active) return;
  const int np4 = lanczos_partials(n_pad);
  lanczos_reduce(in, np4, j, h);
  if (!last && blockIdx.x == 0 && threadIdx.x == 0) {
    st->alpha[j] = h[j];
    st->steps = j + 1;
  }
  const int i = blockIdx.x * LZ_BLOCK + threadIdx.x;
  double t = (double)ld_or0(w, i, i < n_pad);
  for (int v0 = 0; v0 <= j; v0 += 8) {
    float q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = ld_or0(Q, (long long)(v0 + u) * n_pad + i, v0 + u <= j && i < n_pad);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (v0 + u <= j) t -= h[v0 + u] * q[u];
  }
  if (i < n_pad) w[i] = (float)t;
  const double y = (double)(float)t;   // the stored value
  if (!last) {
    lanczos_partial_dots(Q, n_pad, j, i, y, out, np4);
  } else {
    const int wave = threadIdx.x / WAVE, lane = threadIdx.x & (WAVE - 1);
    const double d = wave_sum(y * y);
    if (lane == 0) out[4 * blockIdx.x + wave] = d;
  }
}

__global__ __launch_bounds__(LZ_BLOCK) void lanczos_next_kernel(float* Q, int n_pad, const float* w, int j, int m,
                                                                const double* sq, LanczosState* st) {
  __shared__ double h[1];
  if (j >= st->active || j == m - 1) return;
  lanczos_reduce(sq, lanczos_partials(n_pad), 0, h);
  const double beta = sqrt(h[0]);
  if (beta == 0.0) {
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = j + 1;
    return;
  }
  const int i = blockIdx.x * LZ_BLOCK + threadIdx.x;
  if (i < n_pad) Q[(long long)(j + 1) * n_pad + i] = (float)((double)w[i] / beta);
  if (blockIdx.x == 0 && threadIdx.x == 0) st->beta[j] = beta;
}

// Largest eigenpair of the Lanczos tridiagonal matrix (alpha on the diagonal,
// beta beside it, kk = steps entries) on one wave: the eigenvalue by
// multisection on Sturm counts (the 64 lanes evaluate 64 points of the
// bracket per round, so it shrinks 65-fold; the Gershgorin interval is the
// start), then its eigenvector by two steps of inverse iteration (Gaussian
// elimination with partial pivoting on the tridiagonal matrix, on lane 0).
// Same result as the full eigendecomposition to rounding, without its
// sweeps.
__device__ __forceinline__ int sturm_below(const double* a, const double* b2, int kk, double x, double pivmin) {
  int cnt = 0;
  double q = 1.0;
  for (int i = 0; i < kk; ++i) {
    q = (a[i] - x) - (i > 0 ? b2[i - 1] / q : 0.0);
    if (fabs(q) < pivmin) q = -pivmin;
    cnt += q < 0.0 ? 1 : 0;
  }
  return cnt;
}

__global__ __launch_bounds__(64) void lanczos_top_kernel(LanczosState* st) {
  __shared__ double a[LZ_MAX], b[LZ_MAX], b2[LZ_MAX];
  __shared__ double dg[LZ_MAX], u1[LZ_MAX], u2[LZ_MAX], ml[LZ_MAX], y[LZ_MAX];
  __shared__ int sw[LZ_MAX];
  const int lane = threadIdx.x;
  const int kk = st->steps;
  if (kk < 1) {   // no step taken (cannot happen after lanczos_init): no pair
    if (lane == 0) st->rho = 0.0;
    return;
  }
  for (int i = lane; i < kk; i += WAVE) {
    a[i] = st->alpha[i];
    b[i] = i + 1 < kk ? st->beta[i] : 0.0;
    b2[i] = b[i] * b[i];
  }
  __syncthreads();
  double lo = 1e300, hi = -1e300, bmax = 0.0;
  for (int i = lane; i < kk; i += WAVE) {
    const double r = fabs(b[i]) + (i > 0 ? fabs(b[i - 1]) : 0.0);
    lo = fmin(lo, a[i] - r);
    hi = fmax(hi, a[i] + r);
    bmax = fmax(bmax, b2[i]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = fmin(lo, __shfl_xor(lo, o, WAVE));
    hi = fmax(hi, __shfl_xor(hi, o, WAVE));
    bmax = fmax(bmax, __shfl_xor(bmax, o, WAVE));
  }
  const double pivmin = 0x1p-1000 * fmax(1.0, bmax);
  for (int it = 0; it < 16; ++it) {
    const double w = hi - lo;
    if (!(w > 0x1p-52 * fmax(fabs(lo), fabs(hi)))) break;
    const double x = lo + w * (double)(lane + 1) / 65.0;
    const int c = sturm_below(a, b2, kk, x, pivmin);
    const unsigned long long m = __ballot(c >= kk);
    if (m == 0ull) {
      lo = __shfl(x, WAVE - 1, WAVE);
    } else {
      const int f = __ffsll((long long)m) - 1;
      const double xf = __shfl(x, f, WAVE), xp = __shfl(x, f > 0 ? f - 1 : 0, WAVE);
      hi = xf;
      if (f > 0) lo = xp;
    }
  }
  const double lam = 0.5 * (lo + hi);
  if (lane == 0) {
    // elimination of T - lam I with partial pivoting (rows i, i + 1)
    const double eps = 0x1p-52 * fmax(fabs(lo), fabs(hi)) + pivmin;
    for (int i = 0; i < kk; ++i) {
      dg[i] = a[i] - lam;
      u1[i] = b[i];
      u2[i] = 0.0;
    }
    for (int i = 0; i + 1 < kk; ++i) {
      const double sub = b[i];   // entry (i + 1, i)
      if (fabs(dg[i]) >= fabs(sub)) {
        const double d = dg[i] != 0.0 ? dg[i] : eps;
        dg[i] = d;
        ml[i] = sub / d;
        sw[i] = 0;
        dg[i + 1] -= ml[i] * u1[i];
      } else {
        ml[i] = dg[i] / sub;
        sw[i] = 1;
        const double d1 = dg[i + 1], e1 = u1[i + 1], o1 = u1[i];
        dg[i] = sub;
        u1[i] = d1;
        u2[i] = e1;
        dg[i + 1] = o1 - ml[i] * d1;
        u1[i + 1] = -ml[i] * e1;
      }
    }
    if (dg[kk - 1] == 0.0) dg[kk - 1] = eps;
    for (int i = 0; i < kk; ++i) y[i] = 1.0;
    for (int pass = 0; pass < 2; ++pass) {
      for (int i = 0; i + 1 < kk; ++i) {   // forward: the row operations on y
        if (sw[i]) {
          const double t = y[i];
          y[i] = y[i + 1];
          y[i + 1] = t - ml[i] * y[i];
        } else {
          y[i + 1] -= ml[i] * y[i];
        }
      }
      for (int i = kk - 1; i >= 0; --i) {   // back substitution
        double t = y[i];
        if (i + 1 < kk) t -= u1[i] * y[i + 1];
        if (i + 2 < kk) t -= u2[i] * y[i + 2];
        y[i] = t / dg[i];
      }
      double nrm = 0.0;
      for (int i = 0; i < kk; ++i) nrm += y[i] * y[i];
      nrm = sqrt(nrm);
      for (int i = 0; i < kk; ++i) y[i] /= nrm;
    }
    st->rho = lam;
  }
  __syncthreads();
  for (int i = lane; i < kk; i += WAVE) st->y[i] = y[i];
}

// v = Q y (y from lanczos_top_kernel), one position per thread, every load
// issued before the sum.
__global__ __launch_bounds__(256) void lanczos_vec_kernel(const float* Q, int n_pad, float* v,
                                                          const LanczosState* st) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int kk = st->steps;
  if (i >= n_pad) return;
  double t = 0.0;
  for (int a0 = 0; a0 < kk; a0 += 8) {
    float q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = ld_or0(Q, (long long)(a0 + u) * n_pad + i, a0 + u < kk);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (a0 + u < kk) t += st->y[a0 + u] * (double)q[u];
  }
  v[i] = (float)t;
}

// theta = sqrt(rho + ||B v - rho v||); alpha_x0 = 1 / theta (0 for theta = 0).
__global__ __launch_bounds__(1024) void lanczos_theta_kernel(const float* bv, const float* v, int n_pad,
                                                             const LanczosState* st, float* theta_dev,
                                                             float* alpha_x0, float* theta_user) {
  __shared__ double red[16];
  const int tid = threadIdx.x;
  const double rho = st->rho;
  double acc = 0.0;
  for (int i = tid; i < n_pad; i += 1024) {
    const double d = (double)bv[i] - rho * v[i];
    acc += d * d;
  }
  const double res = sqrt(block_sum(acc, red));
  if (tid == 0) {
    const double t = rho + res;
    const double th = t > 0.0 ? sqrt(t) : 0.0;
    *theta_dev = (float)th;
    *alpha_x0 = th > 0.0 ? (float)(1.0 / th) : 0.f;
    if (theta_user) *theta_user = (float)th;
  }
}

// out = fp16(x), eight elements per thread (n8 groups of eight)
__global__ void to_f16_kernel(const float* __restrict__ x, long long n8, f16_t* __restrict__ out) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n8; i += (long long)gridDim.x * blockDim.x) {
    const u32x4_t lo = ld16(x + 8 * i), hi = ld16(x + 8 * i + 4);
    const u32x4_t h = {pack_h2(__uint_as_float(lo[0]), __uint_as_float(lo[1])),
                       pack_h2(__uint_as_float(lo[2]), __uint_as_float(lo[3])),
                       pack_h2(__uint_as_float(hi[0]), __uint_as_float(hi[1])),
                       pack_h2(__uint_as_float(hi[2]), __uint_as_float(hi[3]))};
    *reinterpret_cast<u32x4_t*>(out + 8 * i) = h;
  }
}

struct PsdPlan {
  int n, k, steps, n_pad, K, lz;
  bool copy_in, quintic, f16;
  bool wide;   // fp16 products on 256 x 256 tiles (n_pad a multiple of 256, at least 4096)
  float *zp, *r, *xa, *xb, *s32, *bm, *c;
  f16_t *xh0, *xh1, *bh, *ah;   // fp16 filter: operand copies of X (current, next), B and (quintic) A
  f16_t* rh;                    // fp16 filter: R / theta, the restore product's operand
  float *vt, *zt, *E, *lam, *ut, *coefR, *coefX, *coefP;
  int* ndef;
  double *part, *fac;
  float *qlan, *w, *t, *v, *theta, *alpha_x0;
  bool frob;       // scale_mode: theta = ||R||_F from the residual pass's tile sums
  float* sumsq;    // [tiles] sums of R^2 per 128 x 128 tile (Frobenius scale)
  LanczosState* lst;
  double* lpart;   // Lanczos step partial sums: two blocks of LZ_MAX rows
  // wide tracked bases (K > PSD_NARROW_MAX): K x K problems in global memory
  bool wk;
  int kp, kr;      // K rounded up to 32 (small matrices), to 128 (panel rows)
  double *wpart, *g64, *hb0, *hb1, *eb0, *eb1, *e64, *lw, *dinv, *q64;
  int* czero;      // CholeskyQR: zero-trace flag
  double *wpart2, *g64b;   // the next basis' CholeskyQR (side stream)
  float* us;       // scaled copy of U for the rank-K GEMMs
  float* qn;       // the next basis, CholQR(Z V), panel rows
  BjState* bst;
  double* bjpart;  // block Jacobi: (off-diagonal, total) sums of squares per H block of a sweep's last round
  float* split;    // fp32 filter products: partial accumulators of a last round cut along K
  long long split_cap;
};

static void plan_psd(PsdPlan& p, Arena& ar) {
  const size_t nn = (size_t)p.n_pad * p.n_pad;
  // partial tiles of a last round cut along K: 1024 of 128 x 128 for the
  // fp32 products (64 MB), 512 of 256 x 256 for the fp16 ones (128 MB); none
  // when even the full product has fewer tiles than a 256-CU device holds
  const long long m128 = p.n_pad / 128;
  p.split_cap = p.f16 ? (p.wide ? 512ll * 256 * 256 : 0) : (m128 * m128 >= 256 ? 1024ll * 128 * 128 : 0);
  p.split = p.split_cap ? ar.take<float>((size_t)p.split_cap) : nullptr;
  p.zp = p.copy_in ? ar.take<float>(nn) : nullptr;
  p.r = ar.take<float>(nn);
  p.xa = ar.take<float>(nn);
  p.xb = ar.take<float>(nn);
  p.s32 = p.quintic ? ar.take<float>(nn) : nullptr;
  p.bm = ar.take<float>(nn);
  p.c = p.bm;   // the restore product reuses B's buffer after the filter
  p.xh0 = p.f16 ? ar.take<f16_t>(nn) : nullptr;
  p.xh1 = p.f16 ? ar.take<f16_t>(nn) : nullptr;
  p.bh = p.f16 ? ar.take<f16_t>(nn) : nullptr;
  p.ah = p.f16 && p.quintic ? ar.take<f16_t>(nn) : nullptr;
  p.rh = p.f16 ? ar.take<f16_t>(nn) : nullptr;
  const int kq = p.K > 0 ? p.K : 1;
  const int kr = p.wk ? p.kr : round_up(kq, 32);
  p.vt = ar.take<float>((size_t)kr * p.n_pad);
  p.zt = ar.take<float>((size_t)kr * p.n_pad);
  p.E = ar.take<float>((size_t)kq * kq);
  p.lam = ar.take<float>(kq);
  p.ut = ar.take<float>((size_t)(p.wk ? kr : kq) * p.n_pad);
  if (p.wk) {
    const size_t kk = (size_t)p.kp * p.kp;
    p.us = ar.take<float>((size_t)kr * p.n_pad);
    p.qn = ar.take<float>((size_t)kr * p.n_pad);
    p.wpart = ar.take<double>(kk * cdiv(p.n_pad, WG_CHUNK));
    p.wpart2 = ar.take<double>(kk * cdiv(p.n_pad, WG_CHUNK));
    p.g64 = ar.take<double>(kk);
    p.g64b = ar.take<double>(kk);
    p.hb0 = ar.take<double>(kk);
    p.hb1 = ar.take<double>(kk);
    p.eb0 = ar.take<double>(kk);
    p.eb1 = ar.take<double>(kk);
    p.e64 = ar.take<double>(kk);
    p.lw = ar.take<double>(kk);
    p.dinv = ar.take<double>((size_t)p.kp * CW);
    p.q64 = ar.take<double>((size_t)p.kp * p.n_pad);
    p.czero = ar.take<int>(1);
    p.bst = ar.take<BjState>(1);
    const size_t pairs = (size_t)p.kp / BJ_B / 2;
    p.bjpart = ar.take<double>(2 * pairs * pairs);
  }
  p.coefR = ar.take<float>(kq);
  p.coefX = ar.take<float>(kq);
  p.coefP = ar.take<float>(kq);
  p.ndef = ar.take<int>(1);
  p.part = ar.take<double>(gram_part_elems(1, p.n_pad, kq, kq, false));
  p.fac = ar.take<double>((size_t)kq * kq);
  p.qlan = ar.take<float>((size_t)(p.lz + 1) * p.n_pad);
  p.w = ar.take<float>(p.n_pad);
  p.t = ar.take<float>(p.n_pad);
  p.v = ar.take<float>(p.n_pad);
  p.theta = ar.take<float>(1);
  p.alpha_x0 = ar.take<float>(1);
  p.sumsq = p.frob ? ar.take<float>((size_t)(p.n_pad / 128) * (p.n_pad / 128)) : nullptr;
  p.lst = ar.take<LanczosState>(1);
  p.lpart = ar.take<double>((size_t)2 * LZ_MAX * lanczos_partials(p.n_pad));
}

static int validate_psd(int n, int k, int steps, const float* X, const float* Qwarm, const float* out,
                        const sd_psd_opts& o) {
  if (n < 1 || k < 0 || k >= n || steps < 0 || steps > 1000 || !X || !out) return SD_ERR_INVALID_ARG;
  if (k > WIDE_MAX) return SD_ERR_UNSUPPORTED;
  if (k > 0 && !Qwarm) return SD_ERR_INVALID_ARG;
  if (o.subspace_iters < 1 || o.subspace_iters > 100) return SD_ERR_INVALID_ARG;
  if (o.lanczos_steps < 1 || o.lanczos_steps > LZ_MAX) return SD_ERR_INVALID_ARG;
  if (!(o.gamma > 0.f) || !(o.tau >= 0.f) || !(o.tau < 1.f)) return SD_ERR_INVALID_ARG;
  if (o.tau > 0.f && (o.window < 1 || o.window > k)) return SD_ERR_INVALID_ARG;
  if (o.poly_degree != 3 && o.poly_degree != 5) return SD_ERR_INVALID_ARG;
  if (o.precision != SD_PREC_F32 && o.precision != SD_PREC_F16) return SD_ERR_INVALID_ARG;
  if (o.scale_mode != SD_SCALE_LANCZOS && o.scale_mode != SD_SCALE_FROBENIUS) return SD_ERR_INVALID_ARG;
  if ((long long)n * n > (1ll << 34)) return SD_ERR_UNSUPPORTED;
  if (k > 0) {
    const char* q0 = reinterpret_cast<const char*>(Qwarm);
    const char* q1 = q0 + (size_t)n * k * sizeof(float);
    const char* x0 = reinterpret_cast<const char*>(X);
    const char* x1 = x0 + (size_t)n * n * sizeof(float);
    const char* o0 = reinterpret_cast<const char*>(out);
    const char* o1 = o0 + (size_t)n * n * sizeof(float);
    if ((q0 < x1 && x0 < q1) || (q0 < o1 && o0 < q1)) return SD_ERR_INVALID_ARG;
  }
  return SD_OK;
}

static void make_psd_plan(PsdPlan& p, int n, int k, int steps, const float* X, const sd_psd_opts& o) {
  p.n = n;
  p.k = k;
  p.K = k;
  p.steps = steps;
  p.n_pad = round_up(n, 128);
  p.lz = o.lanczos_steps < n ? o.lanczos_steps : n;
  p.quintic = o.poly_degree == 5;
  p.f16 = o.precision == SD_PREC_F16;
  p.wide = p.f16 && p.n_pad % 256 == 0 && p.n_pad >= 4096;
  p.frob = o.scale_mode == SD_SCALE_FROBENIUS;
  // bases wider than 32 take the wide path: at K = 64 it measured 7.49
  // against 7.73 ms per ADMM iteration (n = 5000, fp16) for the four-wave
  // one-work-group Jacobi; at K = 32 the one-wave Jacobi is faster (6.61
  // against 6.92 ms)
  p.wk = k > PSD_NARROW_MAX;
  p.kp = round_up(k > 0 ? k : 1, 32);
  p.kr = round_up(k > 0 ? k : 1, 128);
  const bool aligned = X && (reinterpret_cast<uintptr_t>(X) % 16 == 0);
  p.copy_in = p.n != p.n_pad || !aligned;
}

static void lanczos(const PsdPlan& p, const float* R, uint64_t seed, float* theta_user, hipStream_t st) {
  ProfScope ps(SD_STAGE_LANCZOS, st);
  const int np = p.n_pad;
  fill(p.qlan, (long long)(p.lz + 1) * np, 0.f, st);
  hipLaunchKernelGGL(lanczos_init_kernel, dim3(1), dim3(1024), 0, st, p.qlan, p.n, np, p.lz, seed, p.lst);
  const dim3 gg(np / 4), gb(256);
  for (int j = 0; j < p.lz; ++j) {
    hipLaunchKernelGGL(gemv_kernel, gg, gb, 0, st, R, np, np, p.qlan + (long long)j * np, p.t);
    hipLaunchKernelGGL(gemv_kernel, gg, gb, 0, st, R, np, np, p.t, p.w);
    if (np < LZ_MULTI_MIN) {
      hipLaunchKernelGGL(lanczos_step_kernel, dim3(1), dim3(1024), 0, st, p.qlan, np, p.w, j, p.lz, p.lst);
      continue;
    }
    const dim3 lg((np + LZ_BLOCK - 1) / LZ_BLOCK), lb(LZ_BLOCK);
    const long long rows = (long long)lanczos_partials(np) * LZ_MAX;
    hipLaunchKernelGGL(lanczos_dots_kernel, lg, lb, 0, st, p.qlan, np, p.w, j, p.lpart, p.lst);
    hipLaunchKernelGGL(lanczos_pass_kernel, lg, lb, 0, st, p.qlan, np, p.w, j, p.lpart, p.lpart + rows, 0, p.lst);
    hipLaunchKernelGGL(lanczos_pass_kernel, lg, lb, 0, st, p.qlan, np, p.w, j, p.lpart + rows, p.lpart, 1, p.lst);
    hipLaunchKernelGGL(lanczos_next_kernel, lg, lb, 0, st, p.qlan, np, p.w, j, p.lz, p.lpart, p.lst);
  }
  hipLaunchKernelGGL(lanczos_top_kernel, dim3(1), dim3(WAVE), 0, st, p.lst);   // kk <= lz: the run may stop early
  hipLaunchKernelGGL(lanczos_vec_kernel, dim3((np + 255) / 256), dim3(256), 0, st, p.qlan, np, p.v, p.lst);
  hipLaunchKernelGGL(gemv_kernel, gg, gb, 0, st, R, np, np, p.v, p.t);
  hipLaunchKernelGGL(gemv_kernel, gg, gb, 0, st, R, np, np, p.t, p.w);
  hipLaunchKernelGGL(lanczos_theta_kernel, dim3(1), dim3(1024), 0, st, p.w, p.v, np, p.lst, p.theta, p.alpha_x0,
                     theta_user);
}

// theta = ||R||_F from the residual pass's per-tile sums of squares (float64,
// fixed order over the tiles), and alpha = 1 / theta (0 for theta = 0).
__global__ __launch_bounds__(WAVE) void frob_scale_kernel(const float* sumsq, int tiles, float* theta_dev,
                                                          float* alpha_x0, float* theta_user) {
  double acc = 0.0;
  for (int t = threadIdx.x; t < tiles; t += WAVE) acc += (double)sumsq[t];
  acc = wave_sum(acc);
  if (threadIdx.x == 0) {
    const double th = sqrt(acc);
    *theta_dev = (float)th;
    *alpha_x0 = th > 0.0 ? (float)(1.0 / th) : 0.f;
    if (theta_user) *theta_user = (float)th;
  }
}

// ------------------------------------------- wide tracked bases ----------
constexpr int BJ_MAX_SWEEPS = 16;   // block Jacobi sweep cap
constexpr int BJ_TOL_EXP = -40;     // stop at off(H) <= 2^-40 ||H||_F
constexpr int BJ_INNER_ROUNDS = BJ_P - 1;   // one sweep of the pair problem per round

// C = A B^T over the panel rows (kp x kp, float64), SYM: A == B; part: the
// chunk partials' scratch.
static void wide_products(const PsdPlan& p, const float* A, const float* B, bool sym, double* part, double* C,
                          hipStream_t st) {
  const int np = p.n_pad, kp = p.kp, nch = cdiv(np, WG_CHUNK), tk = cdiv(kp, 64);
  const int tiles = sym ? tk * (tk + 1) / 2 : tk * tk;
  const dim3 gr(cdiv(kp * kp, 256));
  if (sym) {
    hipLaunchKernelGGL(wide_gram_kernel<true>, dim3(tiles * nch), dim3(256), 0, st, A, np, B, np, kp, np, part);
    hipLaunchKernelGGL(wide_gram_reduce_kernel<true>, gr, dim3(256), 0, st, part, nch, kp, C);
  } else {
    hipLaunchKernelGGL(wide_gram_kernel<false>, dim3(tiles * nch), dim3(256), 0, st, A, np, B, np, kp, np, part);
    hipLaunchKernelGGL(wide_gram_reduce_kernel<false>, gr, dim3(256), 0, st, part, nch, kp, C);
  }
}

// dst = CholQR(src) (K panel rows; rows K .. kr - 1 of dst written as zero),
// with the partials' scratch `part` and the Gram buffer `g`. src and dst may
// not overlap.
static void cholqr_wide(const PsdPlan& p, const float* src, float* dst, int* status, double* part, double* g,
                        hipStream_t st) {
  ProfScope ps(SD_STAGE_CHOLQR, st);
  const int np = p.n_pad, nbk = cdiv(p.K, CW);
  wide_products(p, src, src, true, part, g, st);
  hipLaunchKernelGGL(chol_wide_kernel, dim3(1), dim3(CF_THREADS), 0, st, g, p.K, p.kp, p.lw, p.dinv, p.czero, status);
  fill(dst + (long long)p.K * np, (long long)(p.kr - p.K) * np, 0.f, st);
  for (int ib = 0; ib < nbk; ++ib)
    hipLaunchKernelGGL(chol_solve_wide_kernel, dim3(np / 64), dim3(256), 0, st, src, np, p.K, p.kp, p.lw, p.dinv,
                       p.czero, ib, p.q64, dst);
}

// Zt = V^T Z^T = (Z V)^T on the float32 MFMA GEMM (Z symmetric: its rows),
// on 64 x 64 tiles: with only kr / 128 tile rows, 128 x 128 tiles would leave
// most CUs idle (K = 250, n = 5000: 80 work-groups; 366 -> 193 us).
static void zv_wide(const PsdPlan& p, const float* z, const float* vt, float* zt, hipStream_t st) {
  ProfScope ps(SD_STAGE_SKETCH, st);
  const int np = p.n_pad;
  GemmShape g{p.kr, np, np, np, np, 0, 0, 1};
  EpiStore es{zt, 0, np};
  launch_gemm<GemmCfg<2, 2, 1, 1>, float, false, false>(vt, z, g, es, st);
}

// out = alpha x + U^T diag(mult c) U over the deflated rows (float32 MFMA,
// K = kp); x may be out.
static void rankk_wide(const PsdPlan& p, const float* coef, float mult, const float* x, const float* alpha,
                       float* out, f16_t* xs16, hipStream_t st) {
  ProfScope ps(SD_STAGE_LOWRANK, st);
  const int np = p.n_pad;
  hipLaunchKernelGGL(scale_rows_kernel, grid1((long long)p.kp * np, 256), dim3(256), 0, st, p.ut, np, coef, p.ndef,
                     mult, p.kp, p.us);
  GemmShape g{np, np, p.kp, np, np, 0, 0, 1};
  EpiAxpyDev e{x, alpha, out, xs16, np};
  launch_gemm<CfgTile128, float, true, false, true>(p.us, p.ut, g, e, st);
}

// Rayleigh-Ritz on the wide basis: H = V^T (Z V) in float64, block Jacobi,
// ordering / gate / coefficients, U = V E.
static void ritz_wide(const PsdPlan& p, const float* vt, const float* zt, const sd_psd_opts& o, hipStream_t st) {
  ProfScope ps(SD_STAGE_SMALL, st);
  const int kp = p.kp, np = p.n_pad, nb = kp / BJ_B, P = nb / 2, rps = nb - 1;
  wide_products(p, vt, zt, false, p.wpart, p.g64, st);
  hipLaunchKernelGGL(bj_init_kernel, dim3(cdiv(kp * kp, 256)), dim3(256), 0, st, p.g64, kp, p.hb0, p.eb0, p.bst);
  const dim3 grid(P * P + P * (kp / BJ_P));
  for (int sweep = 0; sweep < BJ_MAX_SWEEPS; ++sweep) {
    for (int t = 0; t < rps; ++t) {
      const long long g = (long long)sweep * rps + t;
      const bool odd = g & 1;
      const int flags = (t == rps - 1 ? BJ_WRITE_PART : 0) | (t == 0 && sweep > 0 ? BJ_TEST_PART : 0);
      hipLaunchKernelGGL(bj_round_kernel, grid, dim3(128), 0, st, odd ? p.hb1 : p.hb0, odd ? p.hb0 : p.hb1,
                         odd ? p.eb1 : p.eb0, odd ? p.eb0 : p.eb1, kp, nb, t, BJ_INNER_ROUNDS, sweep, flags,
                         BJ_TOL_EXP, p.bjpart, p.bst);
    }
  }
  hipLaunchKernelGGL(bj_final_kernel, dim3(1), dim3(128), 0, st, p.bjpart, P * P, BJ_MAX_SWEEPS, BJ_TOL_EXP, p.bst,
                     o.status_dev);
  hipLaunchKernelGGL(ritz_wide_kernel, dim3(1), dim3(1024), 0, st, p.hb0, p.hb1, p.eb0, p.eb1, rps, p.bst, p.K, kp,
                     o.tau, o.window, o.gamma, p.e64, p.lam, p.ndef, p.coefR, p.coefX, p.coefP, o.ritz_out,
                     o.n_deflated_out, o.n_positive_out);
  hipLaunchKernelGGL(wide_rotate_kernel, dim3(cdiv(kp, 64) * (np / 64)), dim3(256), 0, st, p.e64, kp, vt, np, kp,
                     kp, np, p.ut, np, kp);
}

// Library-owned side stream per device (non-blocking, default priority,
// kept until the process ends) for the wide path's next-basis CholeskyQR,
// which only the final basis write waits for: it runs beside the
// Rayleigh-Ritz step. Enqueues that use it hold `mu`.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  std::mutex mu;
  bool ready = false;
};

static int side_stream(SideStream*& ss) {
  static std::mutex mu;
  static SideStream per_dev[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return SD_ERR_HIP;
  std::lock_guard<std::mutex> g(mu);
  SideStream& d = per_dev[dev];
  if (!d.ready) {
    if (hipStreamCreateWithFlags(&d.s, hipStreamNonBlocking) != hipSuccess) return SD_ERR_HIP;
    if (hipEventCreateWithFlags(&d.fork, hipEventDisableTiming) != hipSuccess) return SD_ERR_HIP;
    if (hipEventCreateWithFlags(&d.join, hipEventDisableTiming) != hipSuccess) return SD_ERR_HIP;
    d.ready = true;
  }
  ss = &d;
  return SD_OK;
}

static int run_psd(const PsdPlan& p, const float* X, float* Qwarm, float* out, const sd_psd_opts& o,
                   hipStream_t st) {
  const int np = p.n_pad, n = p.n, K = p.K;
  const long long nn = (long long)np * np;
  const float* z;
  if (p.copy_in) {
    const int blocks = (np / 32) * (np / 32);
    hipLaunchKernelGGL((canon_copy_kernel<float>), dim3(blocks), dim3(256), 0, st, p.zp, nn, np, np, np, X, nn, n,
                       n, 0, 1);
    z = p.zp;
  } else {
    z = X;
  }
  LowRankArgs la{};
  la.rows_pad = np;
  la.cols_pad = np;
  la.batch = 1;
  la.ldx = np;
  la.ldo = np;
  la.ldl = la.ldr = np;
  SideStream* ss = nullptr;
  std::unique_lock<std::mutex> side_lock;
  if (K > 0 && p.wk) {
    // wide basis: V panel (rows K .. kr - 1 zero), (J - 1) x [Z V, CholQR],
    // Z V, then the next basis CholQR(Z V) on the side stream beside
    // Rayleigh-Ritz and R = Z - U lam U^T (a GEMM); the basis is written
    // back at the end of the call
    const int rc = side_stream(ss);
    if (rc != SD_OK) return rc;
    side_lock = std::unique_lock<std::mutex>(ss->mu);
    fill(p.vt + (long long)K * np, (long long)(p.kr - K) * np, 0.f, st);
    hipLaunchKernelGGL(rows_to_panel_kernel, grid1((long long)K * np, 256), dim3(256), 0, st, Qwarm, K, n, np, p.vt);
    for (int j = 0; j + 1 < o.subspace_iters; ++j) {
      zv_wide(p, z, p.vt, p.zt, st);
      cholqr_wide(p, p.zt, p.vt, o.status_dev, p.wpart, p.g64, st);
    }
    zv_wide(p, z, p.vt, p.zt, st);
    if (hipEventRecord(ss->fork, st) != hipSuccess || hipStreamWaitEvent(ss->s, ss->fork, 0) != hipSuccess)
      return SD_ERR_HIP;
    cholqr_wide(p, p.zt, p.qn, o.status_dev, p.wpart2, p.g64b, ss->s);
    if (hipEventRecord(ss->join, ss->s) != hipSuccess) {
      (void)hipStreamSynchronize(ss->s);   // no join point: the caller may free the workspace on return
      return SD_ERR_HIP;
    }
    ritz_wide(p, p.vt, p.zt, o, st);
    rankk_wide(p, p.coefR, 1.f, z, nullptr, p.r, nullptr, st);
    if (p.frob) hipLaunchKernelGGL(tile_sumsq_kernel, dim3((np / 128) * (np / 128)), dim3(256), 0, st, p.r, np, p.sumsq);
  } else if (K > 0) {
    hipLaunchKernelGGL(rows_to_panel_kernel, grid1((long long)K * np, 256), dim3(256), 0, st, Qwarm, K, n, np, p.vt);
    float* vt = p.vt;
    float* zt = p.zt;
    for (int j = 0; j + 1 < o.subspace_iters; ++j) {
      ts_xw<float>(z, nn, np, np, np, vt, 0, np, K, zt, 0, np, 1, st);
      cholqr(zt, 0, np, K, np, 1, p.part, p.fac, o.status_dev, st);
      float* tmp = vt;
      vt = zt;
      zt = tmp;
    }
    ts_xw<float>(z, nn, np, np, np, vt, 0, np, K, zt, 0, np, 1, st);   // Zt = Z V
    {
      ProfScope ps(SD_STAGE_SMALL, st);
      gram_partials(vt, 0, np, zt, 0, np, K, K, np, false, p.part, 1, st);   // V^T (Z V)
#define SD_RITZ(NPV)                                                                                            \
  hipLaunchKernelGGL(ritz_kernel<NPV>, dim3(1), dim3(SM_THREADS), 0, st, p.part, np / GP_CHUNK, K, o.tau, o.window, \
                     o.gamma, p.E, p.lam, p.ndef, p.coefR, p.coefX, p.coefP, o.ritz_out, o.n_deflated_out,          \
                     o.n_positive_out)
      switch (jacobi_class(K)) {   // K <= PSD_NARROW_MAX: one wave
        case 4: SD_RITZ(4); break;
        case 8: SD_RITZ(8); break;
        case 12: SD_RITZ(12); break;
        default: SD_RITZ(16); break;
      }
#undef SD_RITZ
    }
    rotate(vt, 0, np, p.E, 0, nullptr, 0, p.ut, 0, np, K, K, np, 1, st);
    // R = Z - U diag(lam) U^T
    la.x = z;
    la.L = p.ut;
    la.Rr = p.ut;
    la.coef = p.coefR;
    la.kk = p.ndef;
    la.kmax = K;
    la.alpha = nullptr;
    la.out = p.r;
    la.sumsq = p.sumsq;   // Frobenius scale: tile sums of R^2
    lowrank<float, float>(la, st);
    // next basis: CholQR(Zt), written to the caller's Qwarm now (Z V was the
    // last read of the old basis; nothing after this reads Qwarm)
    cholqr(zt, 0, np, K, np, 1, p.part, p.fac, o.status_dev, st);
    hipLaunchKernelGGL(panel_to_rows_kernel, grid1((long long)n * K, 256), dim3(256), 0, st, zt, np, K, n, Qwarm);
  } else {
    la.x = z;
    la.L = la.Rr = p.ut;
    la.coef = p.coefR;
    la.kk = nullptr;
    la.kconst = 0;
    la.kmax = 1;
    la.out = p.r;
    la.sumsq = p.sumsq;
    lowrank<float, float>(la, st);
    if (o.n_deflated_out) hipLaunchKernelGGL(fill_int_kernel, dim3(1), dim3(64), 0, st, o.n_deflated_out, 1ll, 0);
    if (o.n_positive_out) hipLaunchKernelGGL(fill_int_kernel, dim3(1), dim3(64), 0, st, o.n_positive_out, 1ll, 0);
  }
  la.sumsq = nullptr;
  if (p.frob) {
    const int tiles = (np / 128) * (np / 128);
    hipLaunchKernelGGL(frob_scale_kernel, dim3(1), dim3(WAVE), 0, st, p.sumsq, tiles, p.theta, p.alpha_x0,
                       o.theta_out);
  } else {
    lanczos(p, p.r, o.seed, o.theta_out, st);
  }
  // X0 = R / theta + gamma^-1 U sign(lam) U^T
  if (K > 0 && p.wk) {
    rankk_wide(p, p.coefX, 1.f, p.r, p.alpha_x0, p.xa, p.rh, st);
  } else {
    la.x = p.r;
    la.coef = p.coefX;
    la.alpha = p.alpha_x0;
    la.out = p.xa;
    la.xs16 = p.rh;   // fp16 path: R / theta, the restore product's operand
    lowrank<float, float>(la, st);
    la.xs16 = nullptr;
  }

  float* cur = p.xa;
  float* nxt = p.xb;
  const int nc = (o.poly_degree + 1) / 2;
  if (p.f16) {
    // fp16 products on the direct-to-LDS kernel: every epilogue also writes
    // the fp16 copy of what the next product reads (X, B, A), rounded from
    // the same fp32 value the fp32 buffers hold
    f16_t* hc = p.xh0;
    f16_t* hn = p.xh1;
    // 256 x 256 tiles (epilogues from the MFMA layout) for n_pad a multiple
    // of 256 from 4096 up (measured faster there: fewer operand bytes per
    // flop on these long K loops); 128 x 128 otherwise. The
    // quintic's Gram and A^2 keep 128 (its fp32 A copy is written on, and
    // read back from, the same tiles).
    const bool wide = p.wide;
    const long long n8 = (long long)np * np / 8;
    hipLaunchKernelGGL(to_f16_kernel, grid1(n8, 256), dim3(256), 0, st, cur, n8, hc);
    for (int t = 0; t < p.steps; ++t) {
      const float a = o.poly ? o.poly[nc * t] : 1.5f;
      const float b = o.poly ? o.poly[nc * t + 1] : -0.5f;
      const float c = (o.poly && nc == 3) ? o.poly[nc * t + 2] : 0.f;
      GemmShape g{np, np, np, np, np, nn, nn, 1};
      g.part = p.split;   // a mostly idle last round is cut along K (256 x 256 tiles)
      g.part_cap = p.split_cap;
      EpiGramT<f16_t> eg{};
      eg.stride = nn;
      eg.ld = np;
      if (c != 0.f) {
        eg.out32 = p.s32;   // A, for the b A term
        eg.scale32 = 1.f;
        eg.out16 = p.ah;    // A, the operand of A^2
        eg.scale16 = 1.f;
      } else {
        eg.out32 = nullptr;
        eg.out16 = p.bh;    // B = b A
        eg.scale16 = b;
      }
      {
        ProfScope ps(SD_STAGE_NS_GRAM, st);
        if (wide && c == 0.f) {
          EpiGramT<f16_t, false> ew{};
          ew.out16 = eg.out16;
          ew.scale16 = eg.scale16;
          ew.stride = eg.stride;
          ew.ld = eg.ld;
          launch_gemm_dma<CfgDma256, false, true>(hc, hc, g, ew, st);
        } else if (stream_outputs(nn * ((eg.out32 ? 4 : 0) + (eg.out16 ? 2 : 0)))) {
          launch_gemm_dma<CfgDma128, false, true>(hc, hc, g, eg, st);
        } else {   // small enough to stay cacheable for the next product
          launch_gemm_dma<CfgDma128, false, true>(hc, hc, g, cached_stores(eg), st);
        }
      }
      if (c != 0.f) {
        ProfScope ps(SD_STAGE_NS_POLY, st);
        EpiPoly<f16_t> ep{p.s32, p.bh, b, c, nn, np};
        if (stream_outputs(2 * nn)) launch_gemm_dma<CfgDma128, false, true>(p.ah, p.ah, g, ep, st);
        else launch_gemm_dma<CfgDma128, false, true>(p.ah, p.ah, g, cached_stores(ep), st);
      }
      {
        ProfScope ps(SD_STAGE_NS_UPDATE, st);
        // B X = B X^T: the NT form on rows of X; symmetric tiles
        if (wide) {
          // fp32 and fp16 outputs: 6 bytes per entry
          if (stream_outputs(6 * nn)) {
            EpiUpdateSymNR<f16_t, true> eu{cur, a, nxt, hn, nn, np};
            launch_gemm_dma<CfgDma256, false, true>(p.bh, hc, g, eu, st);
          } else {
            EpiUpdateSymNR<f16_t> eu{cur, a, nxt, hn, nn, np};
            launch_gemm_dma<CfgDma256, false, true>(p.bh, hc, g, eu, st);
          }
        } else {
          EpiUpdateSym<f16_t> eu{cur, a, nxt, hn, nn, np};
          launch_gemm_dma<CfgDma128, false, true>(p.bh, hc, g, eu, st);
        }
      }
      float* tmp = cur;
      cur = nxt;
      nxt = tmp;
      f16_t* th = hc;
      hc = hn;
      hn = th;
    }
  }
  auto sym_gemm = [&](const float* A, const float* B, GemmShape g, const auto& epi) {
    g.part = p.split;   // a mostly idle last round is cut along K
    g.part_cap = p.split_cap;
    launch_gemm<CfgTile128, float, false, true>(A, B, g, epi, st);
  };
  for (int t = 0; t < (p.f16 ? 0 : p.steps); ++t) {
    const float a = o.poly ? o.poly[nc * t] : 1.5f;
    const float b = o.poly ? o.poly[nc * t + 1] : -0.5f;
    const float c = (o.poly && nc == 3) ? o.poly[nc * t + 2] : 0.f;
    GemmShape g{np, np, np, np, np, nn, nn, 1};
    EpiGram eg{};
    eg.stride = nn;
    eg.ld = np;
    if (c != 0.f) {
      eg.out32 = p.s32 ? p.s32 : p.bm;
      eg.scale32 = 1.f;
    } else {
      eg.out32 = p.bm;
      eg.scale32 = b;
    }
    {
      ProfScope ps(SD_STAGE_NS_GRAM, st);
      sym_gemm(cur, cur, g, eg);
    }
    if (c != 0.f) {
      ProfScope ps(SD_STAGE_NS_POLY, st);
      EpiPoly<float> ep{p.s32, p.bm, b, c, nn, np};
      sym_gemm(p.s32, p.s32, g, ep);
    }
    EpiUpdate<float, float> eu{};
    eu.x = cur;
    eu.xstride = nn;
    eu.ldx = np;
    eu.ac = a;
    eu.out = nxt;
    eu.ostride = nn;
    eu.ldo = np;
    {
      ProfScope ps(SD_STAGE_NS_UPDATE, st);
      sym_gemm(p.bm, cur, g, eu);
    }
    float* tmp = cur;
    cur = nxt;
    nxt = tmp;
  }
  // C = R g (g symmetric, so the NT form reads rows of g); fp16 path:
  // C = theta fp16(R / theta) fp16(g), the operands the filter left behind
  ProfScope ps(SD_STAGE_RESTORE, st);
  GemmShape g{np, np, np, np, np, nn, nn, 1};
  if (p.f16 && p.wide) {
    EpiScaleStore<false> es{p.c, p.theta, nn, np};
    g.part = p.split;
    g.part_cap = p.split_cap;
    launch_gemm_dma<CfgDma256, false, false>(p.rh, p.steps % 2 ? p.xh1 : p.xh0, g, es, st);
  } else if (p.f16) {
    EpiScaleStore<> es{p.c, p.theta, nn, np};
    launch_gemm_dma<CfgDma128, false, false>(p.rh, p.steps % 2 ? p.xh1 : p.xh0, g, es, st);
  } else {
    EpiStore es{p.c, nn, np};
    g.part = p.split;
    g.part_cap = p.split_cap;
    launch_gemm<CfgTile128, float, false, false>(p.r, cur, g, es, st);
  }
  const int tiles = (np / 64) * (np / 64);
  if (K > 0 && p.wk) {
    // the head as 2 U max(lam, 0) U^T added to C: the output's (C + C^T) / 4
    // then carries (H + H^T) / 2, exactly symmetric
    rankk_wide(p, p.coefP, 2.f, p.c, nullptr, p.c, nullptr, st);
  }
  const float* ut = (K > 0 && !p.wk) ? p.ut : nullptr;
  const int* kk = (K > 0 && !p.wk) ? p.ndef : nullptr;
  if (K <= 16 || p.wk)
    hipLaunchKernelGGL((psd_out_kernel<16>), dim3(tiles), dim3(256), 0, st, p.r, p.c, np, ut, np, p.coefP, kk, n, np, out);
  else   // narrow: K <= PSD_NARROW_MAX = 32
    hipLaunchKernelGGL((psd_out_kernel<32>), dim3(tiles), dim3(256), 0, st, p.r, p.c, np, ut, np, p.coefP, kk, n, np, out);
  if (ss) {   // wide basis: join the side stream, write the next basis
    if (hipStreamWaitEvent(st, ss->join, 0) != hipSuccess) {
      (void)hipStreamSynchronize(ss->s);
      return SD_ERR_HIP;
    }
    hipLaunchKernelGGL(panel_to_rows_kernel, grid1((long long)n * K, 256), dim3(256), 0, st, p.qn, np, K, n, Qwarm);
  }
  return hip_status();
}

// ------------------------------------------------------------------ ADMM --
// Three-block ADMM (eq:admm_iter) for SDPs with diagonal constraints,
// A X = diag(X): A* y = Diag(y) and A A* = I, so the y-update is elementwise.
// Matrices are n x n, row-major, contiguous.
constexpr int ADMM_BLOCKS = 1024;   // fixed grid of the reducing kernels (fixed summation order)

// y_i = b_i / sigma - (X_ii / sigma + S_ii - C_ii)
__global__ __launch_bounds__(256) void admm_y_kernel(const float* __restrict__ X, const float* __restrict__ S,
                                                     const float* __restrict__ C, const float* __restrict__ b, int n,
                                                     float inv_sigma, float* __restrict__ y) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const long long d = (long long)i * n + i;
  y[i] = b[i] * inv_sigma - (X[d] * inv_sigma + S[d] - C[d]);
}

// Z = C - Diag(y) - X / sigma (row by row: work-group g takes rows g,
// g + gridDim.x, ...; no division per element)
__global__ __launch_bounds__(256) void admm_z_kernel(const float* __restrict__ C, const float* __restrict__ X,
                                                     const float* __restrict__ y, int n, float inv_sigma,
                                                     float* __restrict__ Z) {
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const long long r = (long long)i * n;
    for (int j = threadIdx.x; j < n; j += blockDim.x)
      Z[r + j] = C[r + j] - (i == j ? y[i] : 0.f) - X[r + j] * inv_sigma;
  }
}

// X <- X + sigma (S + Diag(y) - C), and per-block float64 partial sums of
// ||Diag(y) + S - C||_F^2, <C, X_new> and ||diag(X_new) - b||^2.
__global__ __launch_bounds__(256) void admm_x_kernel(float* __restrict__ X, const float* __restrict__ S,
                                                     const float* __restrict__ C, const float* __restrict__ y,
                                                     const float* __restrict__ b, int n, float sigma,
                                                     double* __restrict__ part) {
  __shared__ double red[4];
  double dual = 0.0, cx = 0.0, prim = 0.0;
  for (int i = blockIdx.x; i < n; i += gridDim.x) {   // rows g, g + gridDim.x, ...
    const long long rw = (long long)i * n;
    for (int j = threadIdx.x; j < n; j += blockDim.x) {
      const long long e = rw + j;
      const float r = S[e] + (i == j ? y[i] : 0.f) - C[e];
      const float xn = X[e] + sigma * r;
      X[e] = xn;
      dual += (double)r * r;
      cx += (double)C[e] * xn;
      if (i == j) {
        const double pr = (double)xn - b[i];
        prim += pr * pr;
      }
    }
  }
  dual = block_sum(dual, red);
  cx = block_sum(cx, red);
  prim = block_sum(prim, red);
  if (threadIdx.x == 0) {
    part[3 * blockIdx.x] = dual;
    part[3 * blockIdx.x + 1] = cx;
    part[3 * blockIdx.x + 2] = prim;
  }
}

// ||C||_F^2 partial sums (once per call)
__global__ __launch_bounds__(256) void admm_cnorm_kernel(const float* __restrict__ C, int n, double* __restrict__ part) {
  __shared__ double red[4];
  const long long nn = (long long)n * n;
  double acc = 0.0;
  for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < nn; e += (long long)gridDim.x * blockDim.x)
    acc += (double)C[e] * C[e];
  acc = block_sum(acc, red);
  if (threadIdx.x == 0) part[blockIdx.x] = acc;
}

// Scratch of an ADMM call: Z, the partial sums, then the projection's own
// workspace (planned for Z, which the arena aligns to 256 bytes).
static void admm_plan(PsdPlan& p, Arena& ar, int n, int k, int steps, const sd_psd_opts& o, float** Z = nullptr,
                      double** part = nullptr, double** cpart = nullptr) {
  float* z = ar.take<float>((size_t)n * n);
  double* pa = ar.take<double>(3 * ADMM_BLOCKS);
  double* cp = ar.take<double>(ADMM_BLOCKS);
  // sizing (no base) plans with an aligned stand-in address: same copy-in decision
  make_psd_plan(p, n, k, steps, ar.base ? z : reinterpret_cast<const float*>(uintptr_t(256)), o);
  plan_psd(p, ar);
  if (Z) *Z = z;
  if (part) *part = pa;
  if (cpart) *cpart = cp;
}

// eta: the eigenvalue-free terms of eq:admm_eta from the partial sums. One
// work-group; every sum in one fixed order (deterministic).
__global__ __launch_bounds__(256) void admm_eta_kernel(const double* __restrict__ part, const double* __restrict__ cpart,
                                                       const float* __restrict__ b, const float* __restrict__ y, int n,
                                                       float* __restrict__ eta) {
  __shared__ double red[4];
  const int tid = threadIdx.x;
  double bb = 0.0, by = 0.0;
  for (int i = tid; i < n; i += 256) {
    bb += (double)b[i] * b[i];
    by += (double)b[i] * y[i];
  }
  bb = block_sum(bb, red);
  by = block_sum(by, red);
  // the block partials: thread t adds blocks t, t + 256, ..., then a fixed tree
  double dual = 0.0, cx = 0.0, prim = 0.0, cc = 0.0;
  for (int k = tid; k < ADMM_BLOCKS; k += 256) {
    dual += part[3 * k];
    cx += part[3 * k + 1];
    prim += part[3 * k + 2];
    cc += cpart[k];
  }
  dual = block_sum(dual, red);
  cx = block_sum(cx, red);
  prim = block_sum(prim, red);
  cc = block_sum(cc, red);
  if (tid == 0) {
    const double nb = sqrt(bb), nc = sqrt(cc);
    const double e1 = sqrt(prim) / (1.0 + nb);
    const double e2 = sqrt(dual) / (1.0 + nc);
    const double e3 = fabs(cx - by) / (1.0 + fabs(cx) + fabs(by));
    *eta = (float)fmax(e1, fmax(e2, e3));
  }
}

}  // namespace sd

using namespace sd;

extern "C" {

void sd_psd_opts_default(sd_psd_opts* o) {
  if (!o) return;
  *o = sd_psd_opts{};
  o->subspace_iters = 1;
  o->lanczos_steps = 20;
  o->gamma = 1.1f;
  o->tau = 0.f;
  o->window = 1;
  o->poly_degree = 3;
  o->poly = nullptr;
  o->seed = 0;
}

size_t sd_psd_workspace_bytes(int n, int k, const sd_psd_opts* opts) {
  sd_psd_opts o;
  sd_psd_opts_default(&o);
  if (opts) o = *opts;
  if (n < 1 || k < 0 || k >= n || k > WIDE_MAX) return 0;
  PsdPlan p{};
  make_psd_plan(p, n, k, 0, nullptr, o);
  Arena ar;
  plan_psd(p, ar);
  return ar.off + 256;
}

int sd_psd_project_deflated_ex(int n, int k, int steps, const float* X, float* Qwarm, float* out,
                               const sd_psd_opts* opts, hipStream_t stream) {
  sd_psd_opts o;
  sd_psd_opts_default(&o);
  if (opts) o = *opts;
  int rc = validate_psd(n, k, steps, X, Qwarm, out, o);
  if (rc != SD_OK) return rc;
  PsdPlan p{};
  make_psd_plan(p, n, k, steps, X, o);
  Arena sizing;
  plan_psd(p, sizing);
  Scratch scratch;
  rc = scratch.acquire(o.workspace, o.workspace_bytes, sizing.off + 256, stream);
  if (rc != SD_OK) return rc;
  Arena ar;
  ar.base = reinterpret_cast<char*>(scratch.ptr);
  plan_psd(p, ar);
  rc = run_psd(p, X, Qwarm, out, o, stream);
  scratch.release();
  return rc;
}

int sd_psd_project(int n, int steps, const float* X, float* out, hipStream_t stream) {
  return sd_psd_project_deflated_ex(n, 0, steps, X, nullptr, out, nullptr, stream);
}

int sd_psd_project_deflated(int n, int k, int steps, const float* X, float* Qwarm, float* out,
                            hipStream_t stream) {
  return sd_psd_project_deflated_ex(n, k, steps, X, Qwarm, out, nullptr, stream);
}

const char* sd_status_string(int status) {
  switch (status) {
    case SD_OK: return "ok";
    case SD_ERR_INVALID_ARG: return "invalid argument";
    case SD_ERR_UNSUPPORTED: return "unsupported size or option";
    case SD_ERR_HIP: return "HIP runtime error";
    case SD_ERR_NUMERIC: return "numerical failure";
    case SD_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

int sd_version(void) { return 100; }

void sd_profile_set(unsigned mask) {
  Profiler& p = profiler();
  std::lock_guard<std::mutex> g(p.mu);
  p.mask = mask;
}

int sd_profile_read(int stage, double* total_ms, long long* launches) {
  if (stage < 0 || stage >= SD_STAGE_COUNT) return SD_ERR_INVALID_ARG;
  Profiler& p = profiler();
  std::lock_guard<std::mutex> g(p.mu);
  p.drain();
  if (total_ms) *total_ms = p.total_ms[stage];
  if (launches) *launches = p.launches[stage];
  return SD_OK;
}

size_t sd_admm_workspace_bytes(int n, int k, int steps, const sd_psd_opts* opts) {
  sd_psd_opts o;
  sd_psd_opts_default(&o);
  if (opts) o = *opts;
  if (n < 1 || k < 0 || k >= n || k > WIDE_MAX || steps < 0) return 0;
  PsdPlan p{};
  Arena ar;
  admm_plan(p, ar, n, k, steps, o);
  return ar.off + 256;
}

int sd_admm_diag(int n, int iters, int steps, float sigma, const float* C, const float* b, float* X, float* S,
                 float* y, int k, float* Qwarm, int warmup, const sd_psd_opts* opts, float* eta_out, int* ndef_out,
                 hipStream_t stream) {
  sd_psd_opts o;
  sd_psd_opts_default(&o);
  if (opts) o = *opts;
  if (iters < 0 || warmup < 0 || !(sigma > 0.f) || !C || !b || !X || !S || !y) return SD_ERR_INVALID_ARG;
  // the projection reads Z (library scratch) and writes S
  int rc = validate_psd(n, k, steps, C, Qwarm, S, o);
  if (rc != SD_OK) return rc;
  if (iters == 0) return SD_OK;
  const long long nn = (long long)n * n;
  PsdPlan p{};
  Arena sizing;
  admm_plan(p, sizing, n, k, steps, o);
  Scratch scratch;
  rc = scratch.acquire(o.workspace, o.workspace_bytes, sizing.off + 256, stream);
  if (rc != SD_OK) return rc;
  Arena ar;
  ar.base = reinterpret_cast<char*>(scratch.ptr);
  float* Z;
  double *part, *cpart;
  admm_plan(p, ar, n, k, steps, o, &Z, &part, &cpart);
  const float inv_sigma = 1.f / sigma;
  hipLaunchKernelGGL(admm_cnorm_kernel, dim3(ADMM_BLOCKS), dim3(256), 0, stream, C, n, cpart);
  for (int it = 0; it < iters && rc == SD_OK; ++it) {
    hipLaunchKernelGGL(admm_y_kernel, grid1(n, 256), dim3(256), 0, stream, X, S, C, b, n, inv_sigma, y);
    hipLaunchKernelGGL(admm_z_kernel, dim3(ADMM_BLOCKS), dim3(256), 0, stream, C, X, y, n, inv_sigma, Z);
    sd_psd_opts oi = o;
    if (it < warmup) oi.tau = 1e-30f;   // gate held closed: s_r < tau s_1 cannot hold
    oi.n_deflated_out = ndef_out ? ndef_out + it : nullptr;
    oi.n_positive_out = nullptr;
    oi.theta_out = nullptr;
    oi.ritz_out = nullptr;
    if (k > 0 && it < warmup && oi.window < 1) oi.window = 1;
    rc = run_psd(p, Z, Qwarm, S, oi, stream);
    hipLaunchKernelGGL(admm_x_kernel, dim3(ADMM_BLOCKS), dim3(256), 0, stream, X, S, C, y, b, n, sigma, part);
    if (eta_out)
      hipLaunchKernelGGL(admm_eta_kernel, dim3(1), dim3(256), 0, stream, part, cpart, b, y, n, eta_out + it);
  }
  scratch.release();
  if (rc != SD_OK) return rc;
  return hip_status();
}

void sd_profile_reset(void) {
  Profiler& p = profiler();
  std::lock_guard<std::mutex> g(p.mu);
  p.drain();
  for (int i = 0; i < SD_STAGE_COUNT; ++i) {
    p.total_ms[i] = 0.0;
    p.launches[i] = 0;
  }
}

}  // extern "C"
