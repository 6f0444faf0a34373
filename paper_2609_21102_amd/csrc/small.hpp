// Small dense linear algebra on one work-group per matrix, in float64:
//   * Gram of panel rows (Pt[a][:] . Pt[b][:])
//   * CholeskyQR of a panel (one pass; pivots floored at c u tr(Gram))
//   * symmetric eigendecomposition by cyclic Jacobi with a round-robin
//     (parallel) ordering, used for the thin SVD of the reduced matrix of the
//     randomized SVD, for the Rayleigh-Ritz step and for the Lanczos
//     tridiagonal matrix
//   * rotation of a panel by a small matrix (U = Q E and friends).
#pragma once

#include "common.hpp"

namespace sd {

constexpr int SM_MAX = 64;        // largest panel width / eigenproblem
constexpr int SM_THREADS = 256;
constexpr int SM_CHUNK = 128;     // panel positions staged per pass
constexpr int SM_LD = SM_MAX + 1;

struct SmallLds {
  double h[SM_MAX][SM_LD];
  double e[SM_MAX][SM_LD];
  float cha[SM_MAX][SM_CHUNK + 1];
  float chb[SM_MAX][SM_CHUNK + 1];
  double rot_c[SM_MAX / 2], rot_s[SM_MAX / 2];
  int rot_i[SM_MAX / 2], rot_j[SM_MAX / 2];
  double red[SM_THREADS / WAVE];
  double key[SM_MAX];
  int perm[SM_MAX];
};

// out[a][b] = sum_x A[a][x] B[b][x] for a < ca, b < cb over x < len (len a
// multiple of SM_CHUNK). sym: A == B, only a <= b is summed, then mirrored.
// Each entry is accumulated in position order, so the result is
// deterministic.
static __device__ void panel_gram(SmallLds& s, const float* A, int lda, const float* B, int ldb, int ca,
                           int cb, int len, bool sym) {
  constexpr int IPT = SM_MAX * SM_MAX / SM_THREADS;   // items per thread
  const int tid = threadIdx.x;
  const int items = sym ? ca * (ca + 1) / 2 : ca * cb;
  double acc[IPT];
  int ia[IPT], ib[IPT];
#pragma unroll
  for (int u = 0; u < IPT; ++u) {
    acc[u] = 0.0;
    int p = tid + u * SM_THREADS;
    ia[u] = -1;
    ib[u] = -1;
    if (p < items) {
      if (sym) {
        int a = 0;
        while (p >= ca - a) {
          p -= ca - a;
          ++a;
        }
        ia[u] = a;
        ib[u] = a + p;
      } else {
        ia[u] = p / cb;
        ib[u] = p - ia[u] * cb;
      }
    }
  }
  for (int x0 = 0; x0 < len; x0 += SM_CHUNK) {
    for (int e = tid; e < ca * SM_CHUNK; e += SM_THREADS) {
      const int a = e / SM_CHUNK, x = e - a * SM_CHUNK;
      s.cha[a][x] = A[(long long)a * lda + x0 + x];
    }
    if (!sym)
      for (int e = tid; e < cb * SM_CHUNK; e += SM_THREADS) {
        const int a = e / SM_CHUNK, x = e - a * SM_CHUNK;
        s.chb[a][x] = B[(long long)a * ldb + x0 + x];
      }
    __syncthreads();
    float(*cb_)[SM_CHUNK + 1] = sym ? s.cha : s.chb;
#pragma unroll
    for (int u = 0; u < IPT; ++u) {
      if (ia[u] < 0) continue;
      const float* ra = s.cha[ia[u]];
      const float* rb = cb_[ib[u]];
      double t = acc[u];
      for (int x = 0; x < SM_CHUNK; ++x) t += (double)ra[x] * (double)rb[x];
      acc[u] = t;
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < IPT; ++u) {
    if (ia[u] < 0) continue;
    s.h[ia[u]][ib[u]] = acc[u];
    if (sym) s.h[ib[u]][ia[u]] = acc[u];
  }
  __syncthreads();
}

// ------------------------------------------------------------- Jacobi -----
// Eigendecomposition of the symmetric n x n matrix in s.h. On return the
// eigenvalues are on the diagonal of s.h and s.e holds the eigenvectors as
// columns. Rotations (Golub & Van Loan, sym.schur2) are applied for n/2
// disjoint pairs at a time (circle-method ordering); sweeps stop when the
// off-diagonal mass is below 1e-30 of the total, or after 60 sweeps.
static __device__ void jacobi_eig(SmallLds& s, int n) {
  const int tid = threadIdx.x;
  for (int e = tid; e < n * n; e += SM_THREADS) {
    const int i = e / n, j = e - i * n;
    s.e[i][j] = (i == j) ? 1.0 : 0.0;
  }
  __syncthreads();
  if (n <= 1) return;
  const int N = n + (n & 1);
  const int half = N / 2;
  for (int sweep = 0; sweep < 60; ++sweep) {
    double off = 0.0, tot = 0.0;
    for (int e = tid; e < n * n; e += SM_THREADS) {
      const int i = e / n, j = e - i * n;
      const double v = s.h[i][j] * s.h[i][j];
      tot += v;
      if (i != j) off += v;
    }
    off = block_sum(off, s.red);
    tot = block_sum(tot, s.red);
    if (off <= 1e-30 * tot) break;
    for (int r = 0; r < N - 1; ++r) {
      if (tid < half) {
        const int pa = (tid == 0) ? 0 : ((r + tid - 1) % (N - 1)) + 1;
        const int pb = ((r + N - 2 - tid) % (N - 1)) + 1;
        int i = pa < pb ? pa : pb, j = pa < pb ? pb : pa;
        double c = 1.0, sn = 0.0;
        if (j < n) {
          const double aij = s.h[i][j];
          if (aij != 0.0) {
            const double tau = (s.h[j][j] - s.h[i][i]) / (2.0 * aij);
            double t;
            if (fabs(tau) > 1e150) t = 0.5 / tau;
            else t = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
            c = 1.0 / sqrt(1.0 + t * t);
            sn = t * c;
          }
        } else {
          i = j = -1;
        }
        s.rot_i[tid] = i;
        s.rot_j[tid] = j;
        s.rot_c[tid] = c;
        s.rot_s[tid] = sn;
      }
      __syncthreads();
      // columns: H <- H J, E <- E J
      for (int e = tid; e < n * half; e += SM_THREADS) {
        const int row = e / half, p = e - row * half;
        const int i = s.rot_i[p], j = s.rot_j[p];
        if (i < 0) continue;
        const double c = s.rot_c[p], sn = s.rot_s[p];
        const double hi = s.h[row][i], hj = s.h[row][j];
        s.h[row][i] = c * hi - sn * hj;
        s.h[row][j] = sn * hi + c * hj;
        const double ei = s.e[row][i], ej = s.e[row][j];
        s.e[row][i] = c * ei - sn * ej;
        s.e[row][j] = sn * ei + c * ej;
      }
      __syncthreads();
      // rows: H <- J^T H
      for (int e = tid; e < n * half; e += SM_THREADS) {
        const int col = e / half, p = e - col * half;
        const int i = s.rot_i[p], j = s.rot_j[p];
        if (i < 0) continue;
        const double c = s.rot_c[p], sn = s.rot_s[p];
        const double hi = s.h[i][col], hj = s.h[j][col];
        s.h[i][col] = c * hi - sn * hj;
        s.h[j][col] = sn * hi + c * hj;
      }
      __syncthreads();
    }
  }
}

// Rank of each key under "larger key first, then smaller index": s.perm[rank]
// = index. Keys must be set in s.key[0..n).
static __device__ void sort_desc(SmallLds& s, int n) {
  const int tid = threadIdx.x;
  if (tid < n) {
    const double k = s.key[tid];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const double kj = s.key[j];
      if (kj > k || (kj == k && j < tid)) ++rank;
    }
    s.perm[rank] = tid;
  }
  __syncthreads();
}

// --------------------------------------------------------- CholeskyQR -----
// One work-group per panel; Pt[b] is c x ld (fp32), updated in place.
template <int CM>
__global__ __launch_bounds__(SM_THREADS) void cholqr_kernel(float* Pt, long long sp, int ld, int c,
                                                            int len_pad, int* status) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x;
  float* P = Pt + blockIdx.x * sp;
  panel_gram(s, P, ld, P, ld, c, c, len_pad, true);
  double tr = 0.0;
  for (int a = 0; a < c; ++a) tr += s.h[a][a];
  if (tr == 0.0) {
    for (int e = tid; e < c * len_pad; e += SM_THREADS) {
      const int a = e / len_pad, x = e - a * len_pad;
      P[(long long)a * ld + x] = 0.f;
    }
    return;
  }
  const double floor_ = (double)c * 1.1102230246251565e-16 * tr;
  // right-looking Cholesky: lower factor L in s.h (lower triangle)
  for (int j = 0; j < c; ++j) {
    if (tid == 0) {
      double d = s.h[j][j];
      if (d <= floor_) {
        d = floor_;
        if (status) atomicOr(status, 2);
      }
      s.h[j][j] = sqrt(d);
    }
    __syncthreads();
    for (int i = j + 1 + tid; i < c; i += SM_THREADS) s.h[i][j] /= s.h[j][j];
    __syncthreads();
    const int m = c - j - 1;
    for (int e = tid; e < m * m; e += SM_THREADS) {
      const int i = j + 1 + e / m, k = j + 1 + e % m;
      if (k <= i) s.h[i][k] -= s.h[i][j] * s.h[k][j];
    }
    __syncthreads();
  }
  // Q = P R^-1 with R = L^T: forward substitution per position.
  for (int x = tid; x < len_pad; x += SM_THREADS) {
    double q[CM];
#pragma unroll
    for (int jj = 0; jj < CM; ++jj) {
      if (jj < c) {
        double v = (double)P[(long long)jj * ld + x];
#pragma unroll
        for (int i = 0; i < jj; ++i) v -= q[i] * s.h[jj][i];
        q[jj] = v / s.h[jj][jj];
      }
    }
#pragma unroll
    for (int jj = 0; jj < CM; ++jj)
      if (jj < c) P[(long long)jj * ld + x] = (float)q[jj];
  }
}

// ----------------------------------------------- thin SVD of G (Alg. 3) ---
// G = Pt (rp x ld, rows of Q^T A). Eigen-decompose H = G G^T, order the
// eigenvalues decreasingly, and emit for the leading k: singular values, the
// eigenvector matrix E (rp x k), 1/s (0 for s = 0) and the deflation rank
// (fixed k, or the gate of Alg. 1 when tau > 0) with the subtraction
// coefficients -s_j used by the residual pass.
static __global__ __launch_bounds__(SM_THREADS) void svd_head_kernel(const float* G, long long sg, int ldg,
                                                              int len_pad, int rp, int k, float tau,
                                                              float* E, float* sv, float* inv_sv,
                                                              int* keff, float* coef_a, float* s_user,
                                                              int* keff_user) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x, b = blockIdx.x;
  panel_gram(s, G + b * sg, ldg, nullptr, 0, rp, rp, len_pad, true);
  jacobi_eig(s, rp);
  if (tid < rp) s.key[tid] = s.h[tid][tid];
  __syncthreads();
  sort_desc(s, rp);
  for (int e = tid; e < rp * k; e += SM_THREADS) {
    const int a = e / k, j = e - a * k;
    E[(long long)b * rp * k + e] = (float)s.e[a][s.perm[j]];
  }
  if (tid == 0) {
    double sval[SM_MAX];
    for (int j = 0; j < k; ++j) {
      const double lam = s.h[s.perm[j]][s.perm[j]];
      sval[j] = lam > 0.0 ? sqrt(lam) : 0.0;
    }
    int ke = k;
    if (tau > 0.f) {
      const double thr = (double)tau * sval[0];
      ke = 0;
      if (sval[k - 1] < thr)
        for (int j = 0; j < k; ++j) ke += (sval[j] > thr) ? 1 : 0;
    }
    keff[b] = ke;
    if (keff_user) keff_user[b] = ke;
    for (int j = 0; j < k; ++j) {
      const float sj = (float)sval[j];
      sv[b * k + j] = sj;
      inv_sv[b * k + j] = sval[j] > 0.0 ? (float)(1.0 / sval[j]) : 0.f;
      coef_a[b * k + j] = j < ke ? -sj : 0.f;
      if (s_user) s_user[b * k + j] = sj;
    }
  }
}

// ------------------------------------------- Rayleigh-Ritz (Alg. 2) -------
// T = V^T (Z V) (K x K, symmetrized), T = E diag(lam) E^T, Ritz pairs ordered
// by |lam| descending (ties: larger lam, then lower index). Deflated set I:
// all K (tau = 0) or the gate of Alg. 2 on the magnitudes. Coefficients for
// the residual (-lam), the padded start (sign(lam) / gamma) and the restore
// (max(lam, 0)).
static __global__ __launch_bounds__(SM_THREADS) void ritz_kernel(const float* Vt, const float* Zt, int ld, int len_pad,
                                                          int K, float tau, int window, float gamma, float* E,
                                                          float* lam_sorted, int* ndef, float* coef_r,
                                                          float* coef_x, float* coef_p, float* ritz_user,
                                                          int* ndef_user, int* npos_user) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x;
  panel_gram(s, Vt, ld, Zt, ld, K, K, len_pad, false);
  // symmetrize: T = (T + T^T) / 2
  for (int e = tid; e < K * K; e += SM_THREADS) {
    const int i = e / K, j = e - i * K;
    if (i < j) {
      const double v = 0.5 * (s.h[i][j] + s.h[j][i]);
      s.h[i][j] = v;
      s.h[j][i] = v;
    }
  }
  __syncthreads();
  jacobi_eig(s, K);
  // key: |lam| first, then lam; index ties are broken by sort_desc
  if (tid < K) {
    const double lam = s.h[tid][tid];
    s.key[tid] = fabs(lam);
  }
  __syncthreads();
  if (tid < K) {
    const double k0 = s.key[tid], lam = s.h[tid][tid];
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const double kj = s.key[j], lj = s.h[j][j];
      if (kj > k0 || (kj == k0 && (lj > lam || (lj == lam && j < tid)))) ++rank;
    }
    s.perm[rank] = tid;
  }
  __syncthreads();
  for (int e = tid; e < K * K; e += SM_THREADS) {
    const int a = e / K, j = e - a * K;
    E[e] = (float)s.e[a][s.perm[j]];
  }
  if (tid == 0) {
    double lam[SM_MAX];
    for (int j = 0; j < K; ++j) lam[j] = s.h[s.perm[j]][s.perm[j]];
    int nd = K;
    if (tau > 0.f) {
      const double thr = (double)tau * fabs(lam[0]);
      int r = window < 1 ? 1 : (window > K ? K : window);
      nd = 0;
      if (fabs(lam[r - 1]) < thr)
        for (int j = 0; j < K; ++j) nd += (fabs(lam[j]) > thr) ? 1 : 0;
    }
    int np = 0;
    for (int j = 0; j < K; ++j) {
      const bool on = j < nd;
      const double l = lam[j];
      lam_sorted[j] = (float)l;
      if (ritz_user) ritz_user[j] = (float)l;
      coef_r[j] = on ? (float)(-l) : 0.f;
      coef_x[j] = on ? (float)((l > 0.0 ? 1.0 : (l < 0.0 ? -1.0 : 0.0)) / (double)gamma) : 0.f;
      coef_p[j] = (on && l > 0.0) ? (float)l : 0.f;
      if (on && l > 0.0) ++np;
    }
    *ndef = nd;
    if (ndef_user) *ndef_user = nd;
    if (npos_user) *npos_user = np;
  }
}

// ------------------------------------------------------------- rotate -----
// out[b][j][x] = scale[b][j] * sum_{a < kin} E[b][a][j] in[b][a][x] for
// j < kout, x < len (len a multiple of 128). scale may be null (1).
template <int KM>
__global__ __launch_bounds__(128) void rotate_kernel(const float* in, long long si, int ldi, const float* E,
                                                     long long se, const float* scale, long long ssc,
                                                     float* out, long long so, int ldo, int kin, int kout,
                                                     int len, int batch) {
  __shared__ float es[KM * KM];
  const int per = len / 128;
  const int b = blockIdx.x / per;
  const int x = (blockIdx.x - b * per) * 128 + threadIdx.x;
  for (int e = threadIdx.x; e < kin * kout; e += 128) es[e] = E[b * se + e];
  __syncthreads();
  float v[KM];
#pragma unroll
  for (int a = 0; a < KM; ++a) v[a] = a < kin ? in[b * si + (long long)a * ldi + x] : 0.f;
  for (int j = 0; j < kout; ++j) {
    float acc = 0.f;
#pragma unroll
    for (int a = 0; a < KM; ++a)
      if (a < kin) acc += es[a * kout + j] * v[a];
    const float sc = scale ? scale[b * ssc + j] : 1.f;
    out[b * so + (long long)j * ldo + x] = sc * acc;
  }
}

}  // namespace sd
