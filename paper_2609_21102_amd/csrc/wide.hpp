// Wide tracked bases for the deflated PSD projection (Alg. 2 with the
// paper's basis widths, K = ceil(0.05 n): 250 to 350 columns in its SDP runs,
// Sec. 3.3). The K x K problems no longer fit one work-group's LDS, so this
// path splits them:
//   * float64 products of panel rows (the CholeskyQR Gram Z^T Z and the
//     Rayleigh quotient V^T Z V) over 128-position chunks, reduced in chunk order;
//   * CholeskyQR's factor on one work-group, the K x K matrix in global
//     memory (L2-resident), panels of 16 columns in LDS and registers; the
//     panel Q^T = L^-1 Z^T by block rows of 16 over all positions;
//   * a block Jacobi eigensolver over 8-index blocks: every round pairs the
//     blocks by the circle method and rotates each 16 x 16 pair problem with
//     one sweep of the one-wave Jacobi (the same rotations a scalar cyclic
//     Jacobi would apply in a block ordering), one launch per round; the
//     last round of a sweep leaves per-block sums of squares that the next
//     sweep's first round tests for convergence;
//   * the rotation V E as a float64-accumulated product; the
//     rank-K terms of the residual, the padded start and the restore as
//     float32 MFMA GEMMs with an axpy epilogue (gemm.hpp).
#pragma once

#include "common.hpp"
#include "small.hpp"
#include "gemm.hpp"

namespace sd {

constexpr int WIDE_MAX = 512;     // widest tracked basis of this path
constexpr int WG_CHUNK = 128;     // positions per partial of the float64 products (more chunks: more work-groups)
constexpr int BJ_B = 8;           // block Jacobi: indices per block
constexpr int BJ_P = 2 * BJ_B;    // indices per pair problem

// -------------------------------------------- float64 panel products -----
// part[ch][a][b] = sum over the positions x of chunk ch of A[a][x] B[b][x],
// a, b < kp, in float64 and position order (one thread per output). Tiles of
// 64 x 64 outputs (SYM: upper tiles only, A == B); thread (ty, tx) owns rows
// a0 + ty + 16i and columns b0 + tx + 16j. Grid: tiles * nch; 256 threads.
template <bool SYM>
__global__ __launch_bounds__(256) void wide_gram_kernel(const float* __restrict__ A, int lda,
                                                        const float* __restrict__ B, int ldb, int kp, int len,
                                                        double* __restrict__ part) {
  __shared__ double as[32][65];
  __shared__ double bs[32][65];
  const int tk = cdiv(kp, 64);
  const int ntiles = SYM ? tk * (tk + 1) / 2 : tk * tk;
  const int ch = blockIdx.x / ntiles;
  int t = blockIdx.x - ch * ntiles, ta, tb;
  if (SYM) {
    sym_tile(t, tk, ta, tb);
  } else {
    ta = t / tk;
    tb = t - ta * tk;
  }
  const int a0 = ta * 64, b0 = tb * 64;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int x_begin = ch * WG_CHUNK, x_end = min(len, x_begin + WG_CHUNK);
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int x0 = x_begin; x0 < x_end; x0 += 32) {
    float va[8], vb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + 256 * u, r = e >> 5, x = e & 31;
      va[u] = a0 + r < kp ? A[(long long)(a0 + r) * lda + x0 + x] : 0.f;
      vb[u] = b0 + r < kp ? B[(long long)(b0 + r) * ldb + x0 + x] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + 256 * u, r = e >> 5, x = e & 31;
      as[x][r] = (double)va[u];
      bs[x][r] = (double)vb[u];
    }
    __syncthreads();
#pragma unroll 4
    for (int x = 0; x < 32; ++x) {
      double av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[i] = as[x][ty + 16 * i];
        bv[i] = bs[x][tx + 16 * i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(av[i], bv[j], acc[i][j]);
    }
  }
  double* out = part + (long long)ch * kp * kp;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int a = a0 + ty + 16 * i, b = b0 + tx + 16 * j;
      if (a < kp && b < kp) out[(long long)a * kp + b] = acc[i][j];
    }
}

// C[a][b] = sum of the chunk partials in chunk order (SYM: entries below the
// tile diagonal read their mirror, so C is exactly symmetric: a diagonal
// tile's (a, b) and (b, a) sum the same products in the same order).
template <bool SYM>
__global__ __launch_bounds__(256) void wide_gram_reduce_kernel(const double* __restrict__ part, int nch, int kp,
                                                               double* __restrict__ C) {
  const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
  if (e >= (long long)kp * kp) return;
  int a = (int)(e / kp), b = (int)(e - (long long)a * kp);
  if (SYM && a / 64 > b / 64) {
    const int t = a;
    a = b;
    b = t;
  }
  const long long src = (long long)a * kp + b, step = (long long)kp * kp;
  double t = 0.0;
  for (int c = 0; c < nch; ++c) t += part[c * step + src];
  C[e] = t;
}

// ------------------------------------------------------ CholeskyQR -----
// Factor: Gram = L L^T for the leading c x c block of G (kp x kp, float64),
// right-looking by panels of CW = 16 columns, pivots below c u tr(Gram) raised to
// that floor (flag 2 in status) as in the narrow path. One work-group of 512
// threads; L lives in global memory (L2), the panel in LDS:
//   * the CW x CW diagonal block on one wave, row i in lane i's registers; at
//     step j every lane publishes its entry of column j in LDS and reads the
//     column back (one round trip per step), then updates its own row;
//   * the inverse of the diagonal block, column t in lane t's registers
//     (forward substitution), written to Dinv[jb] for the solve below;
//   * the rows below: one row per thread in registers, P D^-T by forward
//     substitution, kept in LDS for the trailing update (4 x 4 blocks).
// A zero trace sets *zero (the solve then writes a zero panel).
constexpr int CF_THREADS = 512;
constexpr int CW = 16;   // panel width (rows of the solve's blocks)
constexpr int CPS = CW + 1;   // LDS row stride of the panel (odd: rows fall in distinct banks)

__global__ __launch_bounds__(CF_THREADS) void chol_wide_kernel(const double* __restrict__ G, int c, int kp,
                                                               double* __restrict__ L, double* __restrict__ Dinv,
                                                               int* zero, int* status) {
  __shared__ double colv[CW];
  __shared__ double D[CW][CW + 1];
  __shared__ double P[WIDE_MAX * CPS];
  __shared__ double red[CF_THREADS / WAVE];
  const int tid = threadIdx.x;
  double tr = 0.0;
  for (int a = tid; a < c; a += CF_THREADS) tr += G[(long long)a * kp + a];
  tr = block_sum(tr, red);
  for (int i = 0; i < kp; ++i)
    for (int k = tid; k < kp; k += CF_THREADS) L[(long long)i * kp + k] = G[(long long)i * kp + k];
  if (tid == 0) *zero = tr == 0.0;
  __syncthreads();
  if (tr == 0.0) return;
  const double floor_ = (double)c * 1.1102230246251565e-16 * tr;
  bool floored = false;
  for (int j0 = 0; j0 < c; j0 += CW) {
    const int w = min(CW, c - j0);
    if (tid < WAVE) {
      // rows past w are identity rows (unit pivot, no coupling)
      const int lane = tid;
      double h[CW];
#pragma unroll
      for (int k = 0; k < CW; ++k)
        h[k] = (lane < w && k <= lane) ? L[(long long)(j0 + lane) * kp + j0 + k] : (k == lane ? 1.0 : 0.0);
#pragma unroll
      for (int j = 0; j < CW; ++j) {
        if (lane < CW) colv[lane] = h[j];
        wave_sync();
        double cv[CW];
#pragma unroll
        for (int k = j; k < CW; ++k) cv[k] = colv[k];
        wave_sync();
        double d = cv[j];
        if (j < w && d <= floor_) {
          d = floor_;
          floored = true;
        }
        const double piv = sqrt(d), r = 1.0 / piv;
        const double lij = lane > j ? h[j] * r : (lane == j ? piv : 0.0);
        h[j] = lij;
#pragma unroll
        for (int k = j + 1; k < CW; ++k)
          if (lane >= k) h[k] -= lij * (cv[k] * r);
        __builtin_amdgcn_sched_barrier(0);   // keep each step's loads in its step (register pressure)
      }
      if (lane < CW) {
#pragma unroll
        for (int k = 0; k < CW; ++k) {
          D[lane][k] = k <= lane ? h[k] : 0.0;
          if (lane < w && k <= lane) L[(long long)(j0 + lane) * kp + j0 + k] = h[k];
        }
      }
      wave_sync();
      if (lane < CW) {   // column t = lane of the block's inverse
        const int t = lane;
        double x[CW];
#pragma unroll
        for (int i = 0; i < CW; ++i) {
          double v = i == t ? 1.0 : 0.0;
#pragma unroll
          for (int u = 0; u < i; ++u) v -= D[i][u] * x[u];
          x[i] = i < t ? 0.0 : v / D[i][i];
          __builtin_amdgcn_sched_barrier(0);
        }
        double* di = Dinv + (long long)(j0 / CW) * CW * CW;
#pragma unroll
        for (int i = 0; i < CW; ++i) di[i * CW + t] = x[i];
      }
    }
    __syncthreads();
    const int m = c - j0 - w;
    for (int rr = tid; rr < m; rr += CF_THREADS) {
      // this thread's row, solved in place in LDS (column-oriented forward
      // substitution; D is read by every thread alike: broadcast)
      const long long row = (long long)(j0 + w + rr) * kp + j0;
      double* pr = P + rr * CPS;
      for (int t = 0; t < CW; ++t) pr[t] = t < w ? L[row + t] : 0.0;
      for (int t = 0; t < w; ++t) {
        const double v = pr[t] / D[t][t];
        pr[t] = v;
        L[row + t] = v;
        for (int u = t + 1; u < w; ++u) pr[u] -= v * D[u][t];
      }
    }
    __syncthreads();
    // trailing update of the lower triangle, 4 x 4 blocks per thread
    const int nbm = cdiv(m, 4);
    const int nblk = nbm * (nbm + 1) / 2;
    for (int blk = tid; blk < nblk; blk += CF_THREADS) {
      int bi = (int)((sqrt(8.0 * blk + 1.0) - 1.0) * 0.5);
      while (bi * (bi + 1) / 2 > blk) --bi;
      while ((bi + 1) * (bi + 2) / 2 <= blk) ++bi;
      const int bk = blk - bi * (bi + 1) / 2;
      double acc[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[i][k] = 0.0;
      for (int t = 0; t < w; ++t) {
        double pi[4], pk[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pi[i] = 4 * bi + i < m ? P[(4 * bi + i) * CPS + t] : 0.0;
          pk[i] = 4 * bk + i < m ? P[(4 * bk + i) * CPS + t] : 0.0;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int k = 0; k < 4; ++k) acc[i][k] = fma(pi[i], pk[k], acc[i][k]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int ii = 4 * bi + i, kk = 4 * bk + k;
          if (ii < m && kk <= ii) L[(long long)(j0 + w + ii) * kp + j0 + w + kk] -= acc[i][k];
        }
    }
    __syncthreads();
  }
  if (tid == 0 && floored && status) atomicOr(status, 2);
}

// Solve: rows i0 .. i0 + CW - 1 (block ib, i0 = CW ib) of Q^T = L^-1 Z^T,
//   Q_ib = Dinv_ib (Z_ib - sum_{u < i0} L[i0 + r][u] Q[u]),
// by block rows, one launch per block (the blocks before it are done).
// Q64 keeps the float64 rows for the later blocks, Q the float32 rows (rows
// at or past c are not written). Work-group: CW rows x 64 positions; thread
// (r, g) owns row r and positions x0 + 4 g .. + 3. Grid: len / 64; 256 threads.
__global__ __launch_bounds__(256) void chol_solve_wide_kernel(const float* __restrict__ Zt, int ld, int c, int kp,
                                                              const double* __restrict__ L,
                                                              const double* __restrict__ Dinv, const int* zero,
                                                              int ib, double* __restrict__ Q64,
                                                              float* __restrict__ Q) {
  static_assert(CW == 16, "thread layout: 16 rows x 16 position groups");
  __shared__ double ls[CW][33];
  __shared__ double qs[32][65];
  const int tid = threadIdx.x, r = tid >> 4, g = tid & 15;
  const int i0 = CW * ib, x0 = blockIdx.x * 64 + 4 * g;
  const bool live = i0 + r < c;
  double acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = live ? (double)Zt[(long long)(i0 + r) * ld + x0 + j] : 0.0;
  for (int u0 = 0; u0 < i0; u0 += 32) {
    const int uw = min(32, i0 - u0);   // i0 is a multiple of 16: 16 or 32
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = tid + 256 * q, rr = e >> 5, uu = e & 31;
      ls[rr][uu] = (i0 + rr < c && uu < uw) ? L[(long long)(i0 + rr) * kp + u0 + uu] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int e = tid + 256 * q, uu = e >> 6, xx = e & 63;
      qs[uu][xx] = uu < uw ? Q64[(long long)(u0 + uu) * ld + blockIdx.x * 64 + xx] : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int uu = 0; uu < 32; ++uu) {
      const double l = ls[r][uu];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fma(-l, qs[uu][4 * g + j], acc[j]);
    }
    __syncthreads();
  }
  // diagonal block: q = Dinv_ib acc over the block's rows
#pragma unroll
  for (int j = 0; j < 4; ++j) qs[r][4 * g + j] = acc[j];
  __syncthreads();
  const double* di = Dinv + (long long)ib * CW * CW + r * CW;
  double out[4] = {0.0, 0.0, 0.0, 0.0};
  for (int v = 0; v <= r; ++v) {
    const double dv = di[v];
#pragma unroll
    for (int j = 0; j < 4; ++j) out[j] = fma(dv, qs[v][4 * g + j], out[j]);
  }
  if (!live) return;
  const bool z = *zero != 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const double v = z ? 0.0 : out[j];
    Q64[(long long)(i0 + r) * ld + x0 + j] = v;
    Q[(long long)(i0 + r) * ld + x0 + j] = (float)v;
  }
}

// ------------------------------------------------ float64 rotations -----
// out[i][x] = sum_{j < kin} M[j][i] P[j][x] for i < kout (float64, j order,
// rounded once), rows kout .. rows_out - 1 written as zero; len a multiple of
// 64. Used for U = V E (M = E). Tiles of 64 outputs
// x 64 positions; thread (ty, tx) owns rows i0 + ty + 16 ii and positions
// x0 + 4 tx .. + 3. Grid: cdiv(rows_out, 64) * (len / 64); 256 threads.
__global__ __launch_bounds__(256) void wide_rotate_kernel(const double* __restrict__ M, int ldm,
                                                          const float* __restrict__ Pt, int ldp, int kin, int kout,
                                                          int len, float* __restrict__ out, int ldo, int rows_out) {
  __shared__ double ms[16][65];
  __shared__ double ps[16][65];
  const int tpx = len / 64;
  const int ti = blockIdx.x / tpx, txb = blockIdx.x - ti * tpx;
  const int i0 = ti * 64, x0 = txb * 64;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  if (i0 >= kout) {   // zero rows only
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int i = i0 + ty + 16 * ii;
      if (i < rows_out) *reinterpret_cast<float4*>(out + (long long)i * ldo + x0 + 4 * tx) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    return;
  }
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int j0 = 0; j0 < kin; j0 += 16) {
    double mv[4];
    float pv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, j = e >> 6, c = e & 63;
      mv[u] = (j0 + j < kin && i0 + c < kout) ? M[(long long)(j0 + j) * ldm + i0 + c] : 0.0;
      pv[u] = j0 + j < kin ? Pt[(long long)(j0 + j) * ldp + x0 + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, j = e >> 6, c = e & 63;
      ms[j][c] = mv[u];
      ps[j][c] = (double)pv[u];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      double a[4], p[4];
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) a[ii] = ms[j][ty + 16 * ii];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) p[jj] = ps[j][4 * tx + jj];
#pragma unroll
      for (int ii = 0; ii < 4; ++ii)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc[ii][jj] = fma(a[ii], p[jj], acc[ii][jj]);
    }
  }
#pragma unroll
  for (int ii = 0; ii < 4; ++ii) {
    const int i = i0 + ty + 16 * ii;
    if (i < rows_out) {
      const bool v = i < kout;
      *reinterpret_cast<float4*>(out + (long long)i * ldo + x0 + 4 * tx) =
          v ? make_float4((float)acc[ii][0], (float)acc[ii][1], (float)acc[ii][2], (float)acc[ii][3])
            : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

// --------------------------------------------------- block Jacobi --------
struct BjState {
  int done;     // converged (or the sweep cap reached): later launches return at once
  int sweeps;   // sweeps applied when done was set
};

struct PairLds {
  double h[BJ_P][BJ_P + 1];
  double e[BJ_P][BJ_P + 1];
  double h2[BJ_P][BJ_P + 1];
  double e2[BJ_P][BJ_P + 1];
};

// Blocks of pair j in round t of the circle method over nb (even) blocks
// (the ordering of jacobi_eig): over nb - 1 rounds every two blocks meet once.
__device__ __forceinline__ void bj_pair(int t, int j, int nb, int& pa, int& pb) {
  const int m = nb - 1;
  int u = t + j - 1, w = t + m - 1 - j;
  u -= u >= m ? m : 0;
  w -= w >= m ? m : 0;
  pa = j == 0 ? 0 : u + 1;
  pb = w + 1;
}
// Global index of local index l (0 .. BJ_P - 1) of the pair of blocks (pa, pb).
__device__ __forceinline__ int bj_index(int l, int pa, int pb) {
  return l < BJ_B ? BJ_B * pa + l : BJ_B * pb + (l - BJ_B);
}

// H0 = (H + H^T) / 2 (exactly symmetric), E0 = I, solver state reset.
__global__ __launch_bounds__(256) void bj_init_kernel(const double* __restrict__ H, int kp, double* __restrict__ H0,
                                                      double* __restrict__ E0, BjState* st) {
  const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
  if (e == 0) {
    st->done = 0;
    st->sweeps = 0;
  }
  if (e >= (long long)kp * kp) return;
  const int i = (int)(e / kp), j = (int)(e - (long long)i * kp);
  H0[e] = i == j ? H[e] : 0.5 * (H[e] + H[(long long)j * kp + i]);
  E0[e] = i == j ? 1.0 : 0.0;
}

// Entries of the BJ_P x BJ_P pair problem held per lane (one wave) and of a
// BJ_P x BJ_P block held per thread (128 threads).
constexpr int BJ_PE = BJ_P * BJ_P / WAVE;
constexpr int BJ_BE = BJ_P * BJ_P / 128;
static_assert(BJ_PE * WAVE == BJ_P * BJ_P && BJ_BE * 128 == BJ_P * BJ_P, "pair blocks split evenly");

// Lane's entries of the problem of blocks (pa, pb): entry e = lane + WAVE i
// is (l, q) = (e / BJ_P, e % BJ_P).
__device__ __forceinline__ void bj_load_pair(const double* __restrict__ H, int kp, int pa, int pb,
                                             double (&v)[BJ_PE]) {
  const int lane = threadIdx.x & (WAVE - 1);
#pragma unroll
  for (int i = 0; i < BJ_PE; ++i) {
    const int e = lane + WAVE * i, l = e / BJ_P, q = e - l * BJ_P;
    v[i] = H[(long long)bj_index(l, pa, pb) * kp + bj_index(q, pa, pb)];
  }
}

// One wave: the pair problem (from bj_load_pair) into s.h, then `rounds`
// rounds of the one-wave Jacobi (0: until converged); s.e is the accumulated
// rotation J.
__device__ __forceinline__ void bj_solve(const double (&v)[BJ_PE], PairLds& s, int rounds) {
  const int lane = threadIdx.x & (WAVE - 1);
#pragma unroll
  for (int i = 0; i < BJ_PE; ++i) {
    const int e = lane + WAVE * i, l = e / BJ_P, q = e - l * BJ_P;
    s.h[l][q] = v[i];
  }
  wave_sync();
  jacobi_eig_wave<BJ_B>(s, BJ_P, -48, rounds);
}

// Convergence of the block Jacobi after a sweep, from the per-block sums of
// squares (off-diagonal, total) that the sweep's last round wrote, summed in
// one fixed order by a 128-thread work-group (every caller gets the same
// decision): done when the off-diagonal mass is at most 2^(2 tol_exp) of the
// total.
__device__ __forceinline__ bool bj_converged(const double* __restrict__ part, int nparts, int tol_exp,
                                             double* red) {
  double off = 0.0, tot = 0.0;
  for (int i = threadIdx.x; i < nparts; i += 128) {
    off += part[2 * i];
    tot += part[2 * i + 1];
  }
  off = block_sum(off, red);
  tot = block_sum(tot, red);
  return off <= __builtin_amdgcn_ldexp(tot, 2 * tol_exp);
}

// Round flags: BJ_WRITE_PART on the last round of a sweep (every H-block
// work-group writes the sums of squares of its output block to part);
// BJ_TEST_PART on the first round of sweep `sweep` > 0 (every work-group first
// tests the previous sweep's sums and all return when it converged;
// work-group 0 records it in the state, so later launches return at once).
constexpr int BJ_WRITE_PART = 1, BJ_TEST_PART = 2;

// One round: P = nb / 2 pairs. Work-groups 0 .. P^2 - 1 write the H block of
// pairs (a, b), Hout[a][b] = J_a^T Hin[a][b] J_b (wave 0 solves pair a, wave 1
// pair b); the next P * (kp / BJ_P) update BJ_P rows of E on pair a's
// columns, Eout = Ein J_a. Every work-group that needs J_a computes it from the
// same entries in the same order, so all copies agree. Reads Hin/Ein, writes
// Hout/Eout (the caller alternates the buffers). Every global load of a round
// (the state flag, the pair problem, the block to rotate) is issued before
// the first wait, so a round costs one memory round trip before its solve
// instead of three. 128 threads.
__global__ __launch_bounds__(128) void bj_round_kernel(const double* __restrict__ Hin, double* __restrict__ Hout,
                                                       const double* __restrict__ Ein, double* __restrict__ Eout,
                                                       int kp, int nb, int t, int rounds, int sweep, int flags,
                                                       int tol_exp, double* __restrict__ part, BjState* st) {
  __shared__ PairLds sa, sb;
  __shared__ double red[128 / WAVE];
  __shared__ int sdone;
  const int P = nb / 2, nh = P * P;
  const int tid = threadIdx.x, wave = tid / WAVE;
  const int bid = blockIdx.x;
  double pv[BJ_PE], bv[BJ_BE];
  // the state flag reaches every wave through LDS: work-group 0 of a testing
  // round may set it while this work-group runs, and all waves of a
  // work-group must take the same branch
  const auto is_done = [&]() {
    if (tid == 0) sdone = st->done;
    __syncthreads();
    if (sdone) return true;
    if (!(flags & BJ_TEST_PART) || !bj_converged(part, nh, tol_exp, red)) return false;
    if (bid == 0 && tid == 0) {
      st->done = 1;
      st->sweeps = sweep;
    }
    return true;
  };
  if (bid < nh) {
    const int a = bid / P, b = bid - a * P;
    int pa, qa, pb, qb;
    bj_pair(t, a, nb, pa, qa);
    bj_pair(t, b, nb, pb, qb);
    if (wave == 0) bj_load_pair(Hin, kp, pa, qa, pv);
    else bj_load_pair(Hin, kp, pb, qb, pv);
#pragma unroll
    for (int i = 0; i < BJ_BE; ++i) {
      const int e = tid + 128 * i, l = e / BJ_P, q = e - l * BJ_P;
      bv[i] = Hin[(long long)bj_index(l, pa, qa) * kp + bj_index(q, pb, qb)];
    }
    if (is_done()) return;
    if (wave == 0) bj_solve(pv, sa, rounds);
    else if (a != b) bj_solve(pv, sb, rounds);
    __syncthreads();
    const PairLds& jb = a == b ? sa : sb;
#pragma unroll
    for (int i = 0; i < BJ_BE; ++i) {
      const int e = tid + 128 * i, l = e / BJ_P, q = e - l * BJ_P;
      sa.h[l][q] = bv[i];
    }
    __syncthreads();
    for (int e = tid; e < BJ_P * BJ_P; e += 128) {   // T = H_ab J_b
      const int l = e / BJ_P, m = e - l * BJ_P;
      double v = 0.0;
#pragma unroll 8
      for (int q = 0; q < BJ_P; ++q) v = fma(sa.h[l][q], jb.e[q][m], v);
      sa.h2[l][m] = v;
    }
    __syncthreads();
    double off = 0.0, tot = 0.0;
    for (int e = tid; e < BJ_P * BJ_P; e += 128) {   // J_a^T T
      const int l = e / BJ_P, m = e - l * BJ_P;
      double v = 0.0;
#pragma unroll 8
      for (int q = 0; q < BJ_P; ++q) v = fma(sa.e[q][l], sa.h2[q][m], v);
      const int gi = bj_index(l, pa, qa), gj = bj_index(m, pb, qb);
      Hout[(long long)gi * kp + gj] = v;
      tot = fma(v, v, tot);
      off = gi != gj ? fma(v, v, off) : off;
    }
    if (flags & BJ_WRITE_PART) {
      off = block_sum(off, red);
      tot = block_sum(tot, red);
      if (tid == 0) {
        part[2 * bid] = off;
        part[2 * bid + 1] = tot;
      }
    }
    return;
  }
  const int idx = bid - nh;
  const int a = idx % P, r0 = (idx / P) * BJ_P;
  int pa, qa;
  bj_pair(t, a, nb, pa, qa);
  if (wave == 0) bj_load_pair(Hin, kp, pa, qa, pv);
  // rows r0 .. r0 + BJ_P - 1 of E on the pair's columns (r0 + BJ_P <= kp)
#pragma unroll
  for (int i = 0; i < BJ_BE; ++i) {
    const int e = tid + 128 * i, rr = e / BJ_P, q = e - rr * BJ_P;
    bv[i] = Ein[(long long)(r0 + rr) * kp + bj_index(q, pa, qa)];
  }
  if (is_done()) return;
  if (wave == 0) bj_solve(pv, sa, rounds);
  __syncthreads();
  // the E rows staged in sa.h (free once the solve is done)
#pragma unroll
  for (int i = 0; i < BJ_BE; ++i) {
    const int e = tid + 128 * i, rr = e / BJ_P, q = e - rr * BJ_P;
    sa.h[rr][q] = bv[i];
  }
  __syncthreads();
  for (int e = tid; e < BJ_P * BJ_P; e += 128) {
    const int rr = e / BJ_P, m = e - rr * BJ_P;
    double v = 0.0;
#pragma unroll 8
    for (int q = 0; q < BJ_P; ++q) v = fma(sa.h[rr][q], sa.e[q][m], v);
    Eout[(long long)(r0 + rr) * kp + bj_index(m, pa, qa)] = v;
  }
}

// After the last sweep's launches: when no round recorded convergence, test
// the last sweep's sums (flag 8 in status when they have not converged: the
// sweep cap was reached) and record max_sweeps. Round g reads buffer g % 2
// and writes (g + 1) % 2, so after G rounds the current matrices are buffer
// G % 2. One work-group of 128 threads.
__global__ __launch_bounds__(128) void bj_final_kernel(const double* __restrict__ part, int nparts, int max_sweeps,
                                                       int tol_exp, BjState* st, int* status) {
  __shared__ double red[128 / WAVE];
  __shared__ int sdone;
  if (threadIdx.x == 0) sdone = st->done;
  __syncthreads();
  if (sdone) return;
  const bool conv = bj_converged(part, nparts, tol_exp, red);
  if (threadIdx.x == 0) {
    st->done = 1;
    st->sweeps = max_sweeps;
    if (!conv && status) atomicOr(status, 8);
  }
}

// Rayleigh-Ritz finish (as ritz_kernel, from the block Jacobi's result):
// Ritz values lam = diag(H) of the current buffers, ordered by |lam|
// descending (ties: larger lam, then lower index); E64[a][j] = E[a][perm[j]]
// for j < K (zero columns K .. kp - 1); the deflated count (all K, or the
// gate of Alg. 2 with window r) and the coefficients of the residual (-lam),
// the padded start (sign(lam) / gamma) and the restore (max(lam, 0)). One
// work-group; K <= WIDE_MAX.
__global__ __launch_bounds__(1024) void ritz_wide_kernel(const double* __restrict__ H0, const double* __restrict__ H1,
                                                         const double* __restrict__ E0, const double* __restrict__ E1,
                                                         int rounds_per_sweep, const BjState* st, int K, int kp,
                                                         float tau, int window, float gamma,
                                                         double* __restrict__ E64, float* lam_sorted, int* ndef,
                                                         float* coef_r, float* coef_x, float* coef_p, float* ritz_user,
                                                         int* ndef_user, int* npos_user) {
  __shared__ double lam[WIDE_MAX], key[WIDE_MAX];
  __shared__ int perm[WIDE_MAX];
  __shared__ int count;
  const int tid = threadIdx.x;
  const long long g = (long long)st->sweeps * rounds_per_sweep;
  const double* H = (g & 1) ? H1 : H0;
  const double* E = (g & 1) ? E1 : E0;
  if (tid < K) {
    lam[tid] = H[(long long)tid * kp + tid];
    key[tid] = fabs(lam[tid]);
  }
  __syncthreads();
  if (tid < K) {
    // total order (order_key: NaN last), so perm is a permutation: it
    // indexes global memory below
    const double k0 = order_key(key[tid]), l0 = order_key(lam[tid]);
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const double kj = order_key(key[j]), lj = order_key(lam[j]);
      if (kj > k0 || (kj == k0 && (lj > l0 || (lj == l0 && j < tid)))) ++rank;
    }
    perm[rank] = tid;
  }
  __syncthreads();
  for (long long e = tid; e < (long long)kp * kp; e += 1024) {
    const int a = (int)(e / kp), j = (int)(e - (long long)a * kp);
    E64[e] = j < K ? E[(long long)a * kp + perm[j]] : 0.0;
  }
  if (tid == 0) {
    const double l0 = fabs(lam[perm[0]]);
    int nd = K;
    if (tau > 0.f) {
      const double thr = (double)tau * l0;
      const int r = window < 1 ? 1 : (window > K ? K : window);
      nd = 0;
      if (fabs(lam[perm[r - 1]]) < thr)
        for (int j = 0; j < K; ++j) nd += (fabs(lam[perm[j]]) > thr) ? 1 : 0;
    }
    int np = 0;
    for (int j = 0; j < nd; ++j) np += lam[perm[j]] > 0.0 ? 1 : 0;
    *ndef = nd;
    if (ndef_user) *ndef_user = nd;
    if (npos_user) *npos_user = np;
    count = nd;
  }
  __syncthreads();
  const int nd = count;
  if (tid < K) {
    const double l = lam[perm[tid]];
    const bool on = tid < nd;
    lam_sorted[tid] = (float)l;
    if (ritz_user) ritz_user[tid] = (float)l;
    coef_r[tid] = on ? (float)(-l) : 0.f;
    coef_x[tid] = on ? (float)((l > 0.0 ? 1.0 : (l < 0.0 ? -1.0 : 0.0)) / (double)gamma) : 0.f;
    coef_p[tid] = (on && l > 0.0) ? (float)l : 0.f;
  }
}

// --------------------------------------------- rank-K terms as GEMMs -----
// Us[j][x] = mult c[j] U[j][x] for j < kdef (device count), 0 for kdef <= j < rows.
__global__ __launch_bounds__(256) void scale_rows_kernel(const float* __restrict__ U, int ld, const float* __restrict__ c,
                                                         const int* __restrict__ kdef, float mult, int rows,
                                                         float* __restrict__ Us) {
  const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
  if (e >= (long long)rows * ld) return;
  const int j = (int)(e / ld);
  Us[e] = j < *kdef ? (mult * c[j]) * U[e] : 0.f;
}

// Per 128 x 128 tile sums of R^2 (the Frobenius scale's partials, the layout
// of the residual pass's tile sums). Grid: (n_pad / 128)^2; 256 threads.
__global__ __launch_bounds__(256) void tile_sumsq_kernel(const float* __restrict__ R, int ld, float* __restrict__ sumsq) {
  __shared__ float red[4];
  const int tc = ld / 128;
  const int i0 = (blockIdx.x / tc) * 128, n0 = (blockIdx.x % tc) * 128;
  const int rg = threadIdx.x >> 4, cg = threadIdx.x & 15;
  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const float* p = R + (long long)(i0 + rg * 8 + r) * ld + n0 + cg * 8;
    const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int c = 0; c < 8; ++c) ss = fmaf(v[c], v[c], ss);
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) sumsq[blockIdx.x] = ss;
}

}  // namespace sd
