// Small dense linear algebra on one work-group per matrix, in float64:
//   * Gram of panel rows (Pt[a][:] . Pt[b][:]) as float64 partial sums over
//     128-position chunks (many work-groups), reduced in chunk order
//   * CholeskyQR of a panel (one pass; pivots floored at c u tr(Gram)):
//     factor on one wave, triangular apply over many work-groups
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
constexpr int SM_LD = SM_MAX + 1;

struct SmallLds {
  double h[SM_MAX][SM_LD];
  double e[SM_MAX][SM_LD];
  double h2[SM_MAX][SM_LD];       // second buffers: a Jacobi round reads one
  double e2[SM_MAX][SM_LD];       // pair of buffers and writes the other
  double rot_c[SM_MAX], rot_d[SM_MAX];   // per index: coefficient on itself / on its partner
  double red[SM_THREADS / WAVE];
  double key[SM_MAX];
  int perm[SM_MAX];
  int rotated;                    // a rotation was applied in this sweep
};

// ------------------------------------------------------------- Jacobi -----
// Eigendecomposition of the symmetric n x n matrix in s.h. On return the
// eigenvalues are on the diagonal of s.h and s.e holds the eigenvectors as
// columns. Each round rotates n/2 disjoint pairs (circle-method ordering;
// rotation angles as in Golub & Van Loan, sym.schur2) and applies all of them
// in one pass: with R the round's rotation, H' = R^T H R and E' = E R are
// written entry by entry into the second buffers. A pair is skipped when
// h_ij^2 <= 2^-100 |h_ii h_jj| or |h_ij| <= 2^tol_exp ||H||_F (the default
// 2^-48 is below what the rounding of the rotations leaves behind); sweeps
// stop after one that rotates nothing, or after 40.
// The angle is chosen in float32 (the round's serial latency is this chain;
// float64 square roots and divisions made it several times longer) on the
// pair's entries scaled by a power of two, and (c, s) are then renormalized
// in float64 by one Newton step for 1 / sqrt(c^2 + s^2), so every rotation is
// orthogonal to float64 rounding. The annihilated entry is left to the
// rotation (about 1e-7 of its size instead of zero); later sweeps take it out.
__device__ __forceinline__ void jacobi_angle(double aii, double ajj, double aij, double& c, double& sn) {
  const double d = ajj - aii;
  const double m = fmax(fabs(d), fabs(2.0 * aij));
  const int ex = __builtin_amdgcn_frexp_exp(m);   // m = f 2^ex, f in [0.5, 1)
  const float df = (float)__builtin_amdgcn_ldexp(d, -ex), af = (float)__builtin_amdgcn_ldexp(aij, -ex);
  // df^2 + 4 af^2 lies in [0.25, 2]: the raw square root and reciprocal apply
  const float r = __builtin_amdgcn_sqrtf(df * df + 4.f * af * af);
  const float t = (df >= 0.f ? 2.f * af : -2.f * af) * __builtin_amdgcn_rcpf(fabsf(df) + r);
  const float cf = __builtin_amdgcn_rsqf(1.f + t * t);
  c = (double)cf;
  sn = (double)t * c;
  const double q = 1.5 - 0.5 * (c * c + sn * sn);   // Newton step of 1 / sqrt(c^2 + s^2) from 1
  c *= q;
  sn *= q;
}

// Partner of index a in round r of the circle method over N (even) indices:
// index 0 meets 1 + (r - 1) mod (N - 1); indices x + 1, y + 1 (x != y) meet
// when x + y = 2 (r - 1) mod (N - 1); the one with 2x = 2(r - 1) meets 0.
// (No integer division: r and a - 1 lie in [0, N - 2], so y starts in
// [-N, 2N - 6] and two conditional additions and one subtraction reduce it.)
__device__ __forceinline__ int jacobi_partner(int a, int r, int N) {
  const int m = N - 1;
  if (a == 0) return r == 0 ? m : r;
  const int x = a - 1;
  int y = 2 * r - 2 - x;
  y += y < 0 ? m : 0;
  y += y < 0 ? m : 0;
  y -= y >= m ? m : 0;
  return y == x ? 0 : y + 1;
}

static __device__ void jacobi_eig(SmallLds& s, int n, int tol_exp = -48) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int e = tid; e < n * n; e += nt) {
    const int i = e / n, j = e - i * n;
    s.e[i][j] = (i == j) ? 1.0 : 0.0;
  }
  __syncthreads();
  if (n <= 1) return;
  const int N = n + (n & 1);
  const int half = N / 2;
  double fro = 0.0;
  for (int e = tid; e < n * n; e += nt) fro += s.h[e / n][e % n] * s.h[e / n][e % n];
  fro = block_sum(fro, s.red);
  const double abs_floor = __builtin_amdgcn_ldexp(sqrt(fro), tol_exp);
  double(*H)[SM_LD] = s.h;
  double(*E)[SM_LD] = s.e;
  double(*H2)[SM_LD] = s.h2;
  double(*E2)[SM_LD] = s.e2;
  // this thread's entries in the update: column b of rows a0, a0 + rows_per_pass, ...
  const int rows_per_pass = nt / n, b = tid % n;
  const int a0 = tid < rows_per_pass * n ? tid / n : n;
  for (int sweep = 0; sweep < 40; ++sweep) {
    if (tid == 0) s.rotated = 0;
    __syncthreads();
    for (int r = 0; r < N - 1; ++r) {
      if (tid < half) {
        // pair of this thread: 1 + (r + tid - 1) mod (N - 1) (0 for thread 0)
        // and 1 + (r + N - 2 - tid) mod (N - 1); both sums lie in [0, 2N - 4]
        const int m = N - 1;
        int u = r + tid - 1, w = r + m - 1 - tid;
        u -= u >= m ? m : 0;
        w -= w >= m ? m : 0;
        const int pa = tid == 0 ? 0 : u + 1, pb = w + 1;
        const int i = pa < pb ? pa : pb, j = pa < pb ? pb : pa;
        if (j < n) {
          double c = 1.0, sn = 0.0;
          const double aij = H[i][j], aii = H[i][i], ajj = H[j][j];
          if (aij * aij > 0x1p-100 * fabs(aii * ajj) && fabs(aij) > abs_floor) {
            jacobi_angle(aii, ajj, aij, c, sn);
            s.rotated = 1;
          }
          // column i <- c col_i - s col_j ; column j <- s col_i + c col_j
          s.rot_c[i] = c;
          s.rot_d[i] = -sn;
          s.rot_c[j] = c;
          s.rot_d[j] = sn;
        } else if (i < n) {   // paired with the padding index: unchanged
          s.rot_c[i] = 1.0;
          s.rot_d[i] = 0.0;
        }
      }
      __syncthreads();
      for (int a = a0; a < n; a += rows_per_pass) {
        int qa = jacobi_partner(a, r, N), qb = jacobi_partner(b, r, N);
        qa = qa < n ? qa : a;   // paired with the padding index: unchanged
        qb = qb < n ? qb : b;
        const double ca = s.rot_c[a], da = s.rot_d[a], cb = s.rot_c[b], db = s.rot_d[b];
        H2[a][b] = ca * (cb * H[a][b] + db * H[a][qb]) + da * (cb * H[qa][b] + db * H[qa][qb]);
        E2[a][b] = cb * E[a][b] + db * E[a][qb];
      }
      __syncthreads();
      double(*t)[SM_LD] = H;
      H = H2;
      H2 = t;
      t = E;
      E = E2;
      E2 = t;
    }
    const int any = s.rotated;
    __syncthreads();
    if (!any) break;
  }
  if (H != s.h) {
    for (int e = tid; e < n * n; e += nt) {
      const int a = e / n, b = e - a * n;
      s.h[a][b] = H[a][b];
      s.e[a][b] = E[a][b];
    }
    __syncthreads();
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

// ------------------------------------------------------ Gram partials -----
// part[b][chunk][item] = sum over the chunk's 128 positions of A[a][x] B[bb][x]
// for the items of gram_item (upper pairs when sym, all pairs otherwise), in
// float64 and position order. Grid: (len_pad / 128) * batch; 256 threads.
constexpr int GP_CHUNK = 128;

__host__ __device__ inline int gram_items(int ca, int cb, bool sym) { return sym ? ca * (ca + 1) / 2 : ca * cb; }

__device__ __forceinline__ void gram_item(int p, int ca, int cb, bool sym, int& a, int& bb) {
  if (sym) {
    int r = 0;
    while (p >= ca - r) {
      p -= ca - r;
      ++r;
    }
    a = r;
    bb = r + p;
  } else {
    a = p / cb;
    bb = p - a * cb;
  }
}

template <int CM>
__global__ __launch_bounds__(256) void gram_partial_kernel(const float* A, long long sa, int lda, const float* B,
                                                           long long sb, int ldb, int ca, int cb, int len_pad,
                                                           bool sym, double* part, int batch) {
  __shared__ float ta[CM][GP_CHUNK + 1];
  __shared__ float tb[CM][GP_CHUNK + 1];
  const int nch = len_pad / GP_CHUNK;
  const int b = blockIdx.x / nch, ch = blockIdx.x - b * nch;
  const int x0 = ch * GP_CHUNK;
  const float* Ab = A + b * sa;
  for (int e = threadIdx.x; e < ca * GP_CHUNK; e += 256) {
    const int a = e / GP_CHUNK, x = e - a * GP_CHUNK;
    ta[a][x] = Ab[(long long)a * lda + x0 + x];
  }
  if (!sym) {
    const float* Bb = B + b * sb;
    for (int e = threadIdx.x; e < cb * GP_CHUNK; e += 256) {
      const int a = e / GP_CHUNK, x = e - a * GP_CHUNK;
      tb[a][x] = Bb[(long long)a * ldb + x0 + x];
    }
  }
  __syncthreads();
  const int items = gram_items(ca, cb, sym);
  double* out = part + ((long long)b * nch + ch) * items;
  for (int p = threadIdx.x; p < items; p += 256) {
    int a, bb;
    gram_item(p, ca, cb, sym, a, bb);
    const float* ra = ta[a];
    const float* rb = sym ? ta[bb] : tb[bb];
    double t = 0.0;
    for (int x = 0; x < GP_CHUNK; ++x) t += (double)ra[x] * (double)rb[x];
    out[p] = t;
  }
}

// s.h[a][bb] = sum of the chunk partials in chunk order (mirrored when sym).
// Loads are issued 32 chunks at a time (one round trip for up to 4096
// positions); the additions keep chunk order.
static __device__ void gram_reduce(SmallLds& s, const double* part, int nch, int ca, int cb, bool sym) {
  const int items = gram_items(ca, cb, sym);
  for (int p = threadIdx.x; p < items; p += blockDim.x) {
    double t = 0.0;
    int c = 0;
    for (; c + 32 <= nch; c += 32) {
      double v[32];
#pragma unroll
      for (int u = 0; u < 32; ++u) v[u] = part[(long long)(c + u) * items + p];
#pragma unroll
      for (int u = 0; u < 32; ++u) t += v[u];
    }
    for (; c + 8 <= nch; c += 8) {
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = part[(long long)(c + u) * items + p];
#pragma unroll
      for (int u = 0; u < 8; ++u) t += v[u];
    }
    for (; c < nch; ++c) t += part[(long long)c * items + p];
    int a, bb;
    gram_item(p, ca, cb, sym, a, bb);
    s.h[a][bb] = t;
    if (sym) s.h[bb][a] = t;
  }
  __syncthreads();
}

// --------------------------------------------------------- CholeskyQR -----
// Factor: Gram = L L^T (right-looking, pivots floored at c u tr(Gram)); L is
// written to fac[b] (c x c, float64, lower). A zero trace writes L = 0, which
// the apply kernel turns into a zero panel. One wave per panel.
static __global__ __launch_bounds__(64) void chol_factor_kernel(const double* part, int nch, int c, double* fac,
                                                         int* status) {
  __shared__ SmallLds s;
  const int b = blockIdx.x, tid = threadIdx.x;
  gram_reduce(s, part + (long long)b * nch * gram_items(c, c, true), nch, c, c, true);
  double tr = 0.0;
  for (int a = 0; a < c; ++a) tr += s.h[a][a];
  double* L = fac + (long long)b * c * c;
  if (tr == 0.0) {
    for (int e = tid; e < c * c; e += 64) L[e] = 0.0;
    return;
  }
  const double floor_ = (double)c * 1.1102230246251565e-16 * tr;
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
    for (int i = j + 1 + tid; i < c; i += 64) s.h[i][j] /= s.h[j][j];
    __syncthreads();
    const int m = c - j - 1;
    for (int e = tid; e < m * m; e += 64) {
      const int i = j + 1 + e / m, k = j + 1 + e % m;
      if (k <= i) s.h[i][k] -= s.h[i][j] * s.h[k][j];
    }
    __syncthreads();
  }
  for (int e = tid; e < c * c; e += 64) {
    const int i = e / c, k = e - i * c;
    L[e] = k <= i ? s.h[i][k] : 0.0;
  }
}

// The same factorization on one wave with rows in registers (c <= CM <= 32):
// lane i owns row i of the lower triangle; column j takes its pivot from
// lane j and the multipliers L[k][j] by cross-lane broadcasts, so no step
// waits on LDS or a barrier.
template <int CM>
__global__ __launch_bounds__(64) void chol_factor_wave_kernel(const double* part, int nch, int c, double* fac,
                                                             int* status) {
  static_assert(CM <= 32, "one row per lane");
  __shared__ SmallLds s;
  const int b = blockIdx.x, lane = threadIdx.x;
  gram_reduce(s, part + (long long)b * nch * gram_items(c, c, true), nch, c, c, true);
  double h[CM];
#pragma unroll
  for (int k = 0; k < CM; ++k) h[k] = (lane < c && k <= lane) ? s.h[lane][k] : 0.0;
  double dg = 0.0;
#pragma unroll
  for (int k = 0; k < CM; ++k)
    if (k == lane) dg = h[k];
  const double tr = __shfl(wave_sum(dg), 0, WAVE);
  double* L = fac + (long long)b * c * c;
  if (tr == 0.0) {
    for (int e = lane; e < c * c; e += WAVE) L[e] = 0.0;
    return;
  }
  const double floor_ = (double)c * 1.1102230246251565e-16 * tr;
  bool floored = false;
#pragma unroll
  for (int j = 0; j < CM; ++j) {
    if (j < c) {
      double d = __shfl(h[j], j, WAVE);   // pivot: lane j's updated diagonal
      if (d <= floor_) {
        d = floor_;
        floored = true;
      }
      const double piv = sqrt(d), inv = 1.0 / piv;
      const double lij = lane > j ? h[j] * inv : (lane == j ? piv : 0.0);
      h[j] = lij;
#pragma unroll
      for (int k = j + 1; k < CM; ++k) {
        if (k < c) {
          const double lkj = __shfl(lij, k, WAVE);
          if (lane >= k) h[k] -= lij * lkj;
        }
      }
    }
  }
  if (floored && lane == 0 && status) atomicOr(status, 2);
  if (lane < c) {
#pragma unroll
    for (int k = 0; k < CM; ++k)
      if (k < c) L[(long long)lane * c + k] = k <= lane ? h[k] : 0.0;
  }
}

// Apply: Q = P R^-1 with R = L^T, by forward substitution per position, in
// place (plus an optional bf16 copy of Q). Grid: (len_pad / 128) * batch; one
// thread per position.
template <int CM>
__global__ __launch_bounds__(128) void chol_apply_kernel(float* Pt, long long sp, int ld, int c, int len_pad,
                                                         const double* fac, int batch, bf16_t* Pt16) {
  __shared__ double L[CM][CM + 1];
  __shared__ double inv_d[CM];
  const int per = len_pad / 128;
  const int b = blockIdx.x / per;
  const int x = (blockIdx.x - b * per) * 128 + threadIdx.x;
  const double* F = fac + (long long)b * c * c;
  for (int e = threadIdx.x; e < c * c; e += 128) L[e / c][e % c] = F[e];
  __syncthreads();
  if (threadIdx.x < c) inv_d[threadIdx.x] = L[threadIdx.x][threadIdx.x] != 0.0 ? 1.0 / L[threadIdx.x][threadIdx.x] : 0.0;
  __syncthreads();
  float* P = Pt + b * sp;
  double q[CM];
#pragma unroll
  for (int jj = 0; jj < CM; ++jj) {
    if (jj < c) {
      double v = (double)P[(long long)jj * ld + x];
#pragma unroll
      for (int i = 0; i < jj; ++i) v -= q[i] * L[jj][i];
      q[jj] = v * inv_d[jj];
    }
  }
#pragma unroll
  for (int jj = 0; jj < CM; ++jj)
    if (jj < c) P[(long long)jj * ld + x] = (float)q[jj];
  if (Pt16) {   // bf16 copy: the panel as a product operand
    bf16_t* P16 = Pt16 + b * sp;
#pragma unroll
    for (int jj = 0; jj < CM; ++jj)
      if (jj < c) P16[(long long)jj * ld + x] = f2bf((float)q[jj]);
  }
}

// ----------------------------------------------- thin SVD of G (Alg. 3) ---
// From the partials of H = G G^T (G = Q^T A, rp x s): eigen-decompose H, order
// the eigenvalues decreasingly, and emit for the leading k: singular values,
// the eigenvector matrix E (rp x k), 1/s (0 for s = 0), and the deflation
// rank (fixed k, or the gate of Alg. 1 when tau > 0) with the subtraction
// coefficients -s_j used by the residual pass. One work-group per matrix.
static __global__ __launch_bounds__(SM_THREADS) void svd_head_kernel(const double* part, int nch, int rp, int k, float tau,
                                                             float* E, float* sv, float* inv_sv, int* keff,
                                                             float* coef_a, float* s_user, int* keff_user) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x, b = blockIdx.x;
  gram_reduce(s, part + (long long)b * nch * gram_items(rp, rp, true), nch, rp, rp, true);
  // off-diagonal floor 2^-40 ||H||_F: the outputs are float32, and the
  // leading eigenvectors move by at most that over the gap to the rest
  jacobi_eig(s, rp, -40);
  if (tid < rp) s.key[tid] = s.h[tid][tid];
  __syncthreads();
  sort_desc(s, rp);
  for (int e = tid; e < rp * k; e += SM_THREADS) {
    const int a = e / k, j = e - a * k;
    E[(long long)b * rp * k + e] = (float)s.e[a][s.perm[j]];
  }
  if (tid < k) {
    const double lam = s.h[s.perm[tid]][s.perm[tid]];
    s.key[tid] = lam > 0.0 ? sqrt(lam) : 0.0;   // reuse: singular values
  }
  __syncthreads();
  if (tid == 0) {
    int ke = k;
    if (tau > 0.f) {
      const double thr = (double)tau * s.key[0];
      ke = 0;
      if (s.key[k - 1] < thr)
        for (int j = 0; j < k; ++j) ke += (s.key[j] > thr) ? 1 : 0;
    }
    keff[b] = ke;
    if (keff_user) keff_user[b] = ke;
    s.perm[SM_MAX - 1] = ke;
  }
  __syncthreads();
  const int ke = s.perm[SM_MAX - 1];
  if (tid < k) {
    const double sj = s.key[tid];
    sv[b * k + tid] = (float)sj;
    inv_sv[b * k + tid] = sj > 0.0 ? (float)(1.0 / sj) : 0.f;
    coef_a[b * k + tid] = tid < ke ? -(float)sj : 0.f;
    if (s_user) s_user[b * k + tid] = (float)sj;
  }
}

// ------------------------------------------- Rayleigh-Ritz (Alg. 2) -------
// From the partials of T = V^T (Z V) (K x K, symmetrized): T = E diag(lam) E^T,
// Ritz pairs ordered by |lam| descending (ties: larger lam, then lower index).
// Deflated set I: all K (tau = 0) or the gate of Alg. 2 on the magnitudes.
// Coefficients for the residual (-lam), the padded start (sign(lam) / gamma)
// and the restore (max(lam, 0)). One work-group.
static __global__ __launch_bounds__(SM_THREADS) void ritz_kernel(const double* part, int nch, int K, float tau, int window,
                                                         float gamma, float* E, float* lam_sorted, int* ndef,
                                                         float* coef_r, float* coef_x, float* coef_p,
                                                         float* ritz_user, int* ndef_user, int* npos_user) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x;
  gram_reduce(s, part, nch, K, K, false);
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
  if (tid < K) s.key[tid] = fabs(s.h[tid][tid]);
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
    const double l0 = fabs(s.h[s.perm[0]][s.perm[0]]);
    int nd = K;
    if (tau > 0.f) {
      const double thr = (double)tau * l0;
      const int r = window < 1 ? 1 : (window > K ? K : window);
      nd = 0;
      if (fabs(s.h[s.perm[r - 1]][s.perm[r - 1]]) < thr)
        for (int j = 0; j < K; ++j) nd += (fabs(s.h[s.perm[j]][s.perm[j]]) > thr) ? 1 : 0;
    }
    int np = 0;
    for (int j = 0; j < K; ++j) {
      const double l = s.h[s.perm[j]][s.perm[j]];
      if (j < nd && l > 0.0) ++np;
    }
    *ndef = nd;
    if (ndef_user) *ndef_user = nd;
    if (npos_user) *npos_user = np;
    s.perm[SM_MAX - 1] = nd;
  }
  __syncthreads();
  const int nd = s.perm[SM_MAX - 1];
  if (tid < K) {
    const double l = s.h[s.perm[tid]][s.perm[tid]];
    const bool on = tid < nd;
    lam_sorted[tid] = (float)l;
    if (ritz_user) ritz_user[tid] = (float)l;
    coef_r[tid] = on ? (float)(-l) : 0.f;
    coef_x[tid] = on ? (float)((l > 0.0 ? 1.0 : (l < 0.0 ? -1.0 : 0.0)) / (double)gamma) : 0.f;
    coef_p[tid] = (on && l > 0.0) ? (float)l : 0.f;
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
