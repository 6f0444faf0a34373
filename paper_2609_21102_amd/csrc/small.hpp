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
  int count;                      // a count broadcast from thread 0 (deflation rank)
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
__device__ __forceinline__ void jacobi_angle_f(double aii, double ajj, double aij, float& cf, float& tf) {
  const double d = ajj - aii;
  const double m = fmax(fabs(d), fabs(2.0 * aij));
  const int ex = __builtin_amdgcn_frexp_exp(m);   // m = f 2^ex, f in [0.5, 1)
  const float df = (float)__builtin_amdgcn_ldexp(d, -ex), af = (float)__builtin_amdgcn_ldexp(aij, -ex);
  // df^2 + 4 af^2 lies in [0.25, 2]: the raw square root and reciprocal apply
  const float r = __builtin_amdgcn_sqrtf(df * df + 4.f * af * af);
  tf = (df >= 0.f ? 2.f * af : -2.f * af) * __builtin_amdgcn_rcpf(fabsf(df) + r);
  cf = __builtin_amdgcn_rsqf(1.f + tf * tf);
}
// (c, s) in float64 from the float32 cosine and tangent: one Newton step of
// 1 / sqrt(c^2 + s^2) from 1. Every caller that starts from the same (cf, tf)
// gets the same (c, s); (1, 0) stays exactly (1, 0).
__device__ __forceinline__ void jacobi_rot64(float cf, float tf, double& c, double& sn) {
  c = (double)cf;
  sn = (double)tf * c;
  const double q = 1.5 - 0.5 * (c * c + sn * sn);
  c *= q;
  sn *= q;
}
__device__ __forceinline__ void jacobi_angle(double aii, double ajj, double aij, double& c, double& sn) {
  float cf, tf;
  jacobi_angle_f(aii, ajj, aij, cf, tf);
  jacobi_rot64(cf, tf, c, sn);
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

static __device__ __forceinline__ void jacobi_eig(SmallLds& s, int n, int tol_exp = -48) {
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

// ---------------------------------------------------- one-wave Jacobi -----
// The same eigendecomposition for n <= 2 NP <= 32 on one wave, with no
// work-group barrier: the small eigenproblems sit on the critical path of the
// call, so the latency of a round is what counts.
//   * The N = 2 NP indices sit in slots T_p = p and B_p = NP + p. A round
//     rotates the NP disjoint pairs (T_p, B_p) (angles and skip rules as in
//     jacobi_eig), then every slot but T_0 moves one step along the ring
//     T_1 -> ... -> T_{NP-1} -> B_{NP-1} -> ... -> B_0 -> T_1 (circle method:
//     N - 1 consecutive rounds pair every two indices once).
//   * Lane l holds the 2 x 2 blocks (p, q) of H in slot coordinates (rows
//     T_p, B_p; columns T_q, B_q) with p NP + q = l + 64 u, so a round's row
//     and column rotations are both local to the lane. Each lane also holds
//     the diagonal blocks' entries of pairs p and q and chooses their angles
//     itself (every lane holding a pair computes the same angle from the same
//     values), so the angles need no exchange. E (rows: indices, columns:
//     slots) is held as 2 x 2 units (rows 2p, 2p + 1; columns T_q, B_q).
//   * The ring step goes through LDS (s.h2, s.e2): one round trip per round.
//   * Stop after N - 1 consecutive rounds without a rotation (every pair was
//     checked with nothing changed in between), or at the first round without
//     one in which no off-diagonal entry passes the rotation rule (the same
//     values, sooner), or after 40 sweeps (or max_rounds rounds when given: a
//     partial solve whose accumulated rotation is s.e).
//   * S: any LDS struct with h, e, h2, e2 of at least N x N (and red for NW > 1).
// Input: s.h (n x n). Output as jacobi_eig: eigenvalues on the diagonal of
// s.h (off-diagonal entries are left as they were) and eigenvectors as the
// columns of s.e; returns the number of rounds. Only the calling wave may
// touch s meanwhile; wave_sync orders its LDS accesses (a single wave's LDS
// operations complete in order).
// NW > 1 (n <= 64): the same scheme on NW waves (the whole work-group, which
// must have 64 NW threads): lane t of the group holds blocks t + 64 NW u, the
// ring step is ordered by work-group barriers, and the "any rotation" vote is
// taken at the first of them (__syncthreads_or); every lane applies its
// rotations unconditionally, which is exact for a skipped pair ((1, 0)).
__device__ __forceinline__ void wave_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int NP>
__device__ __forceinline__ int jw_slot(int r, int p) { return r ? NP + p : p; }

// Slot whose content moves into slot (r, p) on a ring step.
template <int NP>
__device__ __forceinline__ int jw_src(int r, int p) {
  if (r == 0) return p == 0 ? 0 : (p == 1 ? NP : p - 1);
  return p == NP - 1 ? NP - 1 : NP + p + 1;
}

// Index in slot `slot` after R ring steps from the identity placement.
template <int NP>
__device__ __forceinline__ int jw_index(int slot, int R) {
  if (slot == 0) return 0;
  constexpr int M = 2 * NP - 1;   // ring length
  const int k = slot < NP ? slot - 1 : 3 * NP - 2 - slot;   // ring position
  int k0 = (k - R % M) % M;
  k0 += k0 < 0 ? M : 0;
  return k0 <= NP - 2 ? k0 + 1 : 3 * NP - 2 - k0;
}

template <int NP, int NW = 1, typename S = SmallLds>
__device__ __forceinline__ int jacobi_eig_wave(S& s, int n, int tol_exp, int max_rounds = 0) {
  constexpr int N = 2 * NP, NB = NP * NP, L = WAVE * NW, U = (NB + L - 1) / L;
  static_assert(N <= SM_MAX && U <= 4, "at most four 2 x 2 blocks per lane");
  const int lane = NW == 1 ? (int)(threadIdx.x & (WAVE - 1)) : (int)threadIdx.x;
  double h[U][4], e[U][4];
  double tp[U][3], tq[U][3];   // (H[T][T], H[B][B], H[T][B]) of pairs p and q
  int bp[U], bq[U];
  bool act[U];
  double fro = 0.0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int id = lane + L * u;
    act[u] = id < NB;
    bp[u] = act[u] ? id / NP : 0;
    bq[u] = act[u] ? id - bp[u] * NP : 0;
#pragma unroll
    for (int r1 = 0; r1 < 2; ++r1)
#pragma unroll
      for (int r2 = 0; r2 < 2; ++r2) {
        const int a = jw_slot<NP>(r1, bp[u]), b = jw_slot<NP>(r2, bq[u]);
        const double v = (act[u] && a < n && b < n) ? s.h[a][b] : 0.0;
        h[u][2 * r1 + r2] = v;
        fro += v * v;
        e[u][2 * r1 + r2] = (act[u] && 2 * bp[u] + r1 == b) ? 1.0 : 0.0;
      }
    const int pt = jw_slot<NP>(0, bp[u]), pb = jw_slot<NP>(1, bp[u]);
    const int qt = jw_slot<NP>(0, bq[u]), qb = jw_slot<NP>(1, bq[u]);
    tp[u][0] = pt < n ? s.h[pt][pt] : 0.0;
    tp[u][1] = pb < n ? s.h[pb][pb] : 0.0;
    tp[u][2] = pb < n ? s.h[pt][pb] : 0.0;
    tq[u][0] = qt < n ? s.h[qt][qt] : 0.0;
    tq[u][1] = qb < n ? s.h[qb][qb] : 0.0;
    tq[u][2] = qb < n ? s.h[qt][qb] : 0.0;
  }
  if constexpr (NW == 1) fro = wave_sum(fro);
  else fro = block_sum(fro, s.red);
  const double abs_floor = __builtin_amdgcn_ldexp(sqrt(fro), tol_exp);
  int idle = 0, R = 0;
  const int round_cap = max_rounds > 0 ? max_rounds : 40 * (N - 1);
  // Would the rotation rule fire on any off-diagonal entry this lane holds
  // (the entry with its own two diagonal entries, in either orientation)?
  // When it fires on none in a round that rotated nothing, no later round can
  // rotate either, as the values no longer change: the solve stops there,
  // with the values the remaining idle rounds would have left.
  auto pending = [&]() {
    bool any = false;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int r1 = 0; r1 < 2; ++r1)
#pragma unroll
        for (int r2 = 0; r2 < 2; ++r2) {
          const double x = h[u][2 * r1 + r2], a = tp[u][r1], d = tq[u][r2];
          const bool off = bp[u] != bq[u] || r1 != r2;
          any |= act[u] && off && x * x > 0x1p-100 * fabs(a * d) && fabs(x) > abs_floor;
        }
    return any;
  };
  while (idle < N - 1 && R < round_cap) {
    // every lane chooses the angles of its own pairs p and q from their
    // diagonal blocks (the same inputs give the same angles in every lane)
    bool rot = false;
    double cp[U], sp[U], cq[U], sq[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float cf = 1.f, tf = 0.f, cg = 1.f, tg = 0.f;
      if (tp[u][2] * tp[u][2] > 0x1p-100 * fabs(tp[u][0] * tp[u][1]) && fabs(tp[u][2]) > abs_floor) {
        jacobi_angle_f(tp[u][0], tp[u][1], tp[u][2], cf, tf);
        rot = act[u];
      }
      if (tq[u][2] * tq[u][2] > 0x1p-100 * fabs(tq[u][0] * tq[u][1]) && fabs(tq[u][2]) > abs_floor)
        jacobi_angle_f(tq[u][0], tq[u][1], tq[u][2], cg, tg);
      jacobi_rot64(cf, tf, cp[u], sp[u]);
      jacobi_rot64(cg, tg, cq[u], sq[u]);
    }
    if (NW > 1 || __any(rot)) {   // every pair is some active lane's p
      if constexpr (NW == 1) idle = 0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // columns of pair q: T <- c T - s B, B <- s T + c B; then the rows of pair p
        const double x00 = cq[u] * h[u][0] - sq[u] * h[u][1], x01 = sq[u] * h[u][0] + cq[u] * h[u][1];
        const double x10 = cq[u] * h[u][2] - sq[u] * h[u][3], x11 = sq[u] * h[u][2] + cq[u] * h[u][3];
        h[u][0] = cp[u] * x00 - sp[u] * x10;
        h[u][2] = sp[u] * x00 + cp[u] * x10;
        h[u][1] = cp[u] * x01 - sp[u] * x11;
        h[u][3] = sp[u] * x01 + cp[u] * x11;
        const double y00 = cq[u] * e[u][0] - sq[u] * e[u][1], y01 = sq[u] * e[u][0] + cq[u] * e[u][1];
        const double y10 = cq[u] * e[u][2] - sq[u] * e[u][3], y11 = sq[u] * e[u][2] + cq[u] * e[u][3];
        e[u][0] = y00;
        e[u][1] = y01;
        e[u][2] = y10;
        e[u][3] = y11;
      }
    } else if constexpr (NW == 1) {
      ++idle;
      if (!__any(pending())) break;
    }
    // ring step; each lane also picks up the diagonal blocks of its new p, q
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (act[u])
#pragma unroll
        for (int r1 = 0; r1 < 2; ++r1)
#pragma unroll
          for (int r2 = 0; r2 < 2; ++r2) {
            const int b = jw_slot<NP>(r2, bq[u]);
            s.h2[jw_slot<NP>(r1, bp[u])][b] = h[u][2 * r1 + r2];
            s.e2[2 * bp[u] + r1][b] = e[u][2 * r1 + r2];
          }
    if constexpr (NW == 1) {
      wave_sync();
    } else {
      const bool any = __syncthreads_or(rot);
      idle = any ? 0 : idle + 1;
      // (the skipped pairs' unit rotations left the values as they were)
      if (!any && !__syncthreads_or(pending())) break;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (act[u]) {
#pragma unroll
        for (int r1 = 0; r1 < 2; ++r1)
#pragma unroll
          for (int r2 = 0; r2 < 2; ++r2) {
            const int b = jw_src<NP>(r2, bq[u]);
            h[u][2 * r1 + r2] = s.h2[jw_src<NP>(r1, bp[u])][b];
            e[u][2 * r1 + r2] = s.e2[2 * bp[u] + r1][b];
          }
        const int pt = jw_src<NP>(0, bp[u]), pb = jw_src<NP>(1, bp[u]);
        const int qt = jw_src<NP>(0, bq[u]), qb = jw_src<NP>(1, bq[u]);
        tp[u][0] = s.h2[pt][pt];
        tp[u][1] = s.h2[pb][pb];
        tp[u][2] = s.h2[pt][pb];
        tq[u][0] = s.h2[qt][qt];
        tq[u][1] = s.h2[qb][qb];
        tq[u][2] = s.h2[qt][qb];
      }
    if constexpr (NW == 1) wave_sync();
    else __syncthreads();
    ++R;
  }
  // back to index coordinates: slot -> index after R ring steps
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (act[u])
#pragma unroll
      for (int r2 = 0; r2 < 2; ++r2) {
        const int col = jw_index<NP>(jw_slot<NP>(r2, bq[u]), R);
        if (col < n) {
#pragma unroll
          for (int r1 = 0; r1 < 2; ++r1)
            if (2 * bp[u] + r1 < n) s.e[2 * bp[u] + r1][col] = e[u][2 * r1 + r2];
          if (bp[u] == bq[u]) s.h[col][col] = h[u][3 * r2];
        }
      }
  if constexpr (NW == 1) wave_sync();
  else __syncthreads();
  return R;
}

// jacobi_eig for a whole work-group of SM_THREADS: with 0 < NP <= 16 (n <= 2 NP)
// on its first wave, NP = 32 on all four waves, otherwise block-wide.
template <int NP>
__device__ __forceinline__ void jacobi_eig_any(SmallLds& s, int n, int tol_exp = -48) {
  if constexpr (NP == 0) {
    jacobi_eig(s, n, tol_exp);
  } else if constexpr (NP > 16) {
    static_assert(SM_THREADS == 4 * WAVE, "four waves");
    __syncthreads();
    jacobi_eig_wave<NP, 4>(s, n, tol_exp);
    __syncthreads();
  } else {
    __syncthreads();
    if (threadIdx.x < WAVE) jacobi_eig_wave<NP>(s, n, tol_exp);
    __syncthreads();
  }
}
// Wave size class of an n x n eigenproblem (0: block-wide solver).
__host__ __device__ inline int jacobi_class(int n) {
  return n <= 8 ? 4 : n <= 16 ? 8 : n <= 24 ? 12 : n <= 32 ? 16 : n <= 64 ? 32 : 0;
}

// Sort keys of a descending order with NaN last: every comparison of the
// rank loops below is then a total order, so the ranks form a permutation of
// 0 .. n - 1 whatever the values (a NaN compares false both ways and would
// give several entries one rank, leaving slots of perm unwritten).
__device__ __forceinline__ double order_key(double v) { return v == v ? v : -__builtin_inf(); }

// Rank of each key under "larger key first, then smaller index": s.perm[rank]
// = index. Keys must be set in s.key[0..n).
static __device__ __forceinline__ void sort_desc(SmallLds& s, int n) {
  const int tid = threadIdx.x;
  if (tid < n) {
    const double k = order_key(s.key[tid]);
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const double kj = order_key(s.key[j]);
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
  // every load of the chunk is issued before the first LDS store
  constexpr int PER = CM * GP_CHUNK / 256;
  const float* Ab = A + b * sa;
  const float* Bb = B + b * sb;
  float va[PER], vb[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u, a = e / GP_CHUNK, x = e - a * GP_CHUNK;
    va[u] = a < ca ? Ab[(long long)a * lda + x0 + x] : 0.f;
    vb[u] = (!sym && a < cb) ? Bb[(long long)a * ldb + x0 + x] : 0.f;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u, a = e / GP_CHUNK, x = e - a * GP_CHUNK;
    ta[a][x] = va[u];
    if (!sym) tb[a][x] = vb[u];
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

// The symmetric case (A = B) with the same results: the chunk's rows are
// converted to float64 once, into LDS (the product of two float32 values is
// exact in float64, so converting per product or per value gives the same
// terms), and each thread forms a BS x BS block of entries (a, bb) of the
// upper block triangle, every entry one running sum over the positions in
// order, as above. The blocks share their row loads and give BS^2
// independent sums per thread. Grid: (len_pad / 128) * batch; 256 threads;
// CM / BS = 16 block rows (136 blocks). Used for panels of 17 to 64 rows.
template <int CM, int BS>
__global__ __launch_bounds__(256) void gram_partial_sym_kernel(const float* A, long long sa, int lda, int ca,
                                                               int len_pad, double* part, int batch) {
  constexpr int PD = GP_CHUNK + 2;   // doubles per row: rows start 16 bytes apart in the banks
  constexpr int NB = CM / BS, NBLK = NB * (NB + 1) / 2;
  static_assert(NBLK <= 256 && GP_CHUNK % 2 == 0, "one block per thread");
  __shared__ __attribute__((aligned(16))) double td[CM][PD];
  const int nch = len_pad / GP_CHUNK;
  const int b = blockIdx.x / nch, ch = blockIdx.x - b * nch;
  const int x0 = ch * GP_CHUNK;
  constexpr int PER = CM * GP_CHUNK / 256;
  const float* Ab = A + b * sa;
  float va[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u, a = e / GP_CHUNK, x = e - a * GP_CHUNK;
    va[u] = a < ca ? Ab[(long long)a * lda + x0 + x] : 0.f;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = threadIdx.x + 256 * u, a = e / GP_CHUNK, x = e - a * GP_CHUNK;
    td[a][x] = (double)va[u];
  }
  __syncthreads();
  const int blk = threadIdx.x;
  if (blk >= NBLK) return;
  int I = 0, q = blk;   // block (I, J), I <= J, row-major over the upper block triangle
  while (q >= NB - I) {
    q -= NB - I;
    ++I;
  }
  const int J = I + q;
  if (I * BS >= ca || J * BS >= ca) return;
  double t[BS][BS];
#pragma unroll
  for (int i = 0; i < BS; ++i)
#pragma unroll
    for (int j = 0; j < BS; ++j) t[i][j] = 0.0;
#pragma unroll 4
  for (int x = 0; x < GP_CHUNK; x += 2) {
    f64x2_t ra[BS], rb[BS];   // positions x and x + 1 of the block's rows
#pragma unroll
    for (int i = 0; i < BS; ++i) ra[i] = *reinterpret_cast<const f64x2_t*>(&td[I * BS + i][x]);
#pragma unroll
    for (int j = 0; j < BS; ++j) rb[j] = *reinterpret_cast<const f64x2_t*>(&td[J * BS + j][x]);
#pragma unroll
    for (int i = 0; i < BS; ++i)
#pragma unroll
      for (int j = 0; j < BS; ++j) {
        t[i][j] += ra[i][0] * rb[j][0];
        t[i][j] += ra[i][1] * rb[j][1];
      }
  }
  const int items = gram_items(ca, ca, true);
  double* out = part + ((long long)b * nch + ch) * items;
#pragma unroll
  for (int i = 0; i < BS; ++i)
#pragma unroll
    for (int j = 0; j < BS; ++j) {
      const int a = I * BS + i, bb = J * BS + j;
      if (a <= bb && bb < ca) out[a * ca - a * (a - 1) / 2 + (bb - a)] = t[i][j];
    }
}

// s.h[a][bb] = sum of the chunk partials in chunk order (mirrored when sym).
// Loads are issued 32 chunks at a time (one round trip for up to 4096
// positions); the additions keep chunk order.
static __device__ __forceinline__ void gram_reduce(SmallLds& s, const double* part, int nch, int ca, int cb, bool sym) {
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
// the apply kernel turns into a zero panel. One work-group (four waves) per
// panel: all of them reduce the partials and update the trailing triangle.
static __global__ __launch_bounds__(256) void chol_factor_kernel(const double* part, int nch, int c, double* fac,
                                                          int* status) {
  __shared__ SmallLds s;
  const int b = blockIdx.x, tid = threadIdx.x, nt = blockDim.x;
  const int lane = tid & (WAVE - 1), w = tid / WAVE, nw = nt / WAVE;
  gram_reduce(s, part + (long long)b * nch * gram_items(c, c, true), nch, c, c, true);
  double tr = 0.0;
  for (int a = 0; a < c; ++a) tr += s.h[a][a];
  double* L = fac + (long long)b * c * c;
  if (tr == 0.0) {
    for (int e = tid; e < c * c; e += nt) L[e] = 0.0;
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
    for (int i = j + 1 + tid; i < c; i += nt) s.h[i][j] /= s.h[j][j];
    __syncthreads();
    // trailing update of the lower triangle: wave w takes rows j + 1 + w,
    // j + 1 + w + nw, ...; lane l column j + 1 + l (c <= 64 = one wave)
    const int k = j + 1 + lane;
    for (int i = j + 1 + w; i < c; i += nw)
      if (k <= i) s.h[i][k] -= s.h[i][j] * s.h[k][j];
    __syncthreads();
  }
  for (int e = tid; e < c * c; e += nt) {
    const int i = e / c, k = e - i * c;
    L[e] = k <= i ? s.h[i][k] : 0.0;
  }
}

// Split bf16 copy of column x of a panel of c rows (stride sp16): hi rows
// 0 .. c - 1, lo rows c .. 2c - 1, zero rows 2c .. c16 - 1.
template <int CM>
__device__ __forceinline__ void store_split16(bf16_t* P16, int ld, int c, int c16, int x, const double (&q)[CM]) {
#pragma unroll
  for (int jj = 0; jj < CM; ++jj)
    if (jj < c) {
      const float v = (float)q[jj];
      const bf16_t hi = f2bf(v);
      P16[(long long)jj * ld + x] = hi;
      P16[(long long)(c + jj) * ld + x] = f2bf(v - bf2f(hi));
    }
  for (int jj = 2 * c; jj < c16; ++jj) P16[(long long)jj * ld + x] = 0;
}

// Apply: Q = P R^-1 with R = L^T, by forward substitution per position, in
// place (plus an optional split bf16 copy of Q, [batch][c16][ld], stride
// sp16). Grid: (len_pad / 128) * batch; one thread per position.
template <int CM>
__global__ __launch_bounds__(128) void chol_apply_kernel(float* Pt, long long sp, int ld, int c, int len_pad,
                                                         const double* fac, int batch, bf16_t* Pt16, int c16,
                                                         long long sp16) {
  __shared__ __attribute__((aligned(16))) double L[CM][CM + 2];   // even pitch: 16-byte pairs
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
      for (int i = 0; i + 1 < jj; i += 2) {   // the same terms in the same order, two per LDS read
        const f64x2_t l2 = *reinterpret_cast<const f64x2_t*>(&L[jj][i]);
        v -= q[i] * l2[0];
        v -= q[i + 1] * l2[1];
      }
      if (jj & 1) v -= q[jj - 1] * L[jj][jj - 1];
      q[jj] = v * inv_d[jj];
    }
  }
#pragma unroll
  for (int jj = 0; jj < CM; ++jj)
    if (jj < c) P[(long long)jj * ld + x] = (float)q[jj];
  if (Pt16) store_split16<CM>(Pt16 + b * sp16, ld, c, c16, x, q);   // the panel as a product operand
}

// Factor and apply in one launch (c <= CM <= 16). Every work-group reduces the
// partials, factors Gram = L L^T on its first wave and applies Q = P R^-1
// (R = L^T) to its 128 positions, so no work-group waits for another; all of
// them compute the same L from the same partials in the same order.
//   * Factor: lane i holds row i of the lower triangle in registers; at step
//     j every lane publishes its entry of column j in LDS and reads the column
//     back, so one LDS round trip gives every lane the pivot and the
//     multipliers L[k][j] = G'[k][j] / sqrt(pivot), computed alike in every
//     lane. 1 / sqrt(pivot) is the hardware estimate with one Newton step
//     (within an ulp or two of float64 rounding).
//   * Pivots below c u tr(Gram) are raised to it (flag 2 in status, set by
//     the matrix's first work-group); a zero trace gives a zero panel.
//   * Apply: forward substitution per position, in place, plus an optional
//     split bf16 copy of Q (store_split16; [batch][c16][ld], stride sp16).
// Grid: (len_pad / 128) * batch; 128 threads.
template <int CM>
__global__ __launch_bounds__(128) void chol_qr_kernel(float* Pt, long long sp, int ld, int c, int len_pad,
                                                      const double* part, int nch, int* status, bf16_t* Pt16,
                                                      int c16, long long sp16) {
  static_assert(CM <= 16, "rows in registers: wider panels use the two-kernel path");
  __shared__ double G[CM][CM + 1];
  __shared__ __attribute__((aligned(16))) double L[CM][CM + 2];   // even pitch: 16-byte pairs
  __shared__ double inv_d[CM];
  __shared__ double colv[CM];
  const int per = len_pad / 128;
  const int b = blockIdx.x / per, tile = blockIdx.x - b * per;
  const int tid = threadIdx.x;
  // this thread's panel column, loaded first: its latency overlaps the
  // reduction and the factorization
  const int x = tile * 128 + tid;
  float* P = Pt + b * sp;
  float pv[CM];
#pragma unroll
  for (int jj = 0; jj < CM; ++jj) pv[jj] = jj < c ? P[(long long)jj * ld + x] : 0.f;
  // Gram from the chunk partials, in chunk order
  {
    const int items = c * (c + 1) / 2;
    const double* pb = part + (long long)b * nch * items;
    for (int q = tid; q < items; q += 128) {
      double t = 0.0;
      int ch = 0;
      for (; ch + 8 <= nch; ch += 8) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = pb[(long long)(ch + u) * items + q];
#pragma unroll
        for (int u = 0; u < 8; ++u) t += v[u];
      }
      for (; ch < nch; ++ch) t += pb[(long long)ch * items + q];
      int a, bb;
      gram_item(q, c, c, true, a, bb);
      G[a][bb] = t;
      G[bb][a] = t;
    }
  }
  __syncthreads();
  if (tid < WAVE) {
    // The Gram is padded to CM x CM with tr(Gram) on the diagonal past c
    // (above the floor, and independent of the leading block), so every loop
    // below has compile-time bounds.
    const int lane = tid;
    double tr = 0.0;
#pragma unroll
    for (int k = 0; k < CM; ++k)
      if (k < c) tr += G[k][k];
    const double floor_ = (double)c * 1.1102230246251565e-16 * tr;
    double h[CM];
#pragma unroll
    for (int k = 0; k < CM; ++k)
      h[k] = (lane < c && k <= lane) ? G[lane][k] : (k == lane ? tr : 0.0);
    bool floored = false;
    if (tr == 0.0) {   // zero panel: L = 0 and zero reciprocals
#pragma unroll
      for (int k = 0; k < CM; ++k) h[k] = 0.0;
      if (lane < CM) inv_d[lane] = 0.0;
    } else {
#pragma unroll
      for (int j = 0; j < CM; ++j) {
        // column j (lane i: entry (i, j) of the updated matrix) through LDS;
        // every lane then forms the pivot and the multipliers itself
        if (lane < CM) colv[lane] = h[j];
        wave_sync();
        double cv[CM];
#pragma unroll
        for (int k = j; k < CM; ++k) cv[k] = colv[k];
        wave_sync();
        double d = cv[j];
        if (d <= floor_) {
          d = floor_;
          floored = true;
        }
        double r = __builtin_amdgcn_rsq(d);
        r = r * (1.5 - 0.5 * d * r * r);
        const double lij = lane > j ? h[j] * r : (lane == j ? d * r : 0.0);
        h[j] = lij;
        if (lane == j) inv_d[j] = r;
#pragma unroll
        for (int k = j + 1; k < CM; ++k)
          if (lane >= k) h[k] -= lij * (cv[k] * r);
      }
    }
    if (lane < CM) {
#pragma unroll
      for (int k = 0; k < CM; ++k) L[lane][k] = h[k];
    }
    if (floored && lane == 0 && tile == 0 && status) atomicOr(status, 2);
  }
  __syncthreads();
  // (the runtime bound keeps the compiler from hoisting all of L's reads)
  double q[CM];
#pragma unroll
  for (int jj = 0; jj < CM; ++jj) {
    if (jj < c) {
      double v = (double)pv[jj];
#pragma unroll
      for (int i = 0; i + 1 < jj; i += 2) {   // the same terms in the same order, two per LDS read
        const f64x2_t l2 = *reinterpret_cast<const f64x2_t*>(&L[jj][i]);
        v -= q[i] * l2[0];
        v -= q[i + 1] * l2[1];
      }
      if (jj & 1) v -= q[jj - 1] * L[jj][jj - 1];
      q[jj] = v * inv_d[jj];
    }
  }
#pragma unroll
  for (int jj = 0; jj < CM; ++jj)
    if (jj < c) P[(long long)jj * ld + x] = (float)q[jj];
  if (Pt16) store_split16<CM>(Pt16 + b * sp16, ld, c, c16, x, q);   // the panel as a product operand
}

// ----------------------------------------------- thin SVD of G (Alg. 3) ---
// From the partials of H = G G^T (G = Q^T A, rp x s), in float64: eigen-
// decompose H, order the eigenvalues decreasingly, and emit for the leading
// k: singular values, the eigenvector matrix E (rp x k), 1/s (0 for s = 0),
// the deflation rank (fixed: kcap = k; or the gate of Alg. 1 when tau > 0
// over the window of k estimated values, min(kcap, max{i : s_i > tau s_1})
// when s_k < tau s_1, else 0) and the subtraction coefficients -s_j used by
// the residual pass. One work-group per matrix; NP = jacobi_class(rp). The
// factors U and V follow in head_factors_kernel.
template <int NP>
__global__ __launch_bounds__(SM_THREADS) void svd_head_kernel(const double* part, int nch, int rp, int k, int kcap,
                                                              float tau,
                                                              double* E, float* sv, float* inv_sv, int* keff,
                                                              float* coef_a, float* s_user, int* keff_user) {
  __shared__ SmallLds s;
  const int tid = threadIdx.x, b = blockIdx.x;
  gram_reduce(s, part + (long long)b * nch * gram_items(rp, rp, true), nch, rp, rp, true);
  // off-diagonal floor 2^-40 ||H||_F: the outputs are float32, and the
  // leading eigenvectors move by at most that over the gap to the rest
  jacobi_eig_any<NP>(s, rp, -40);
  if (tid < rp) s.key[tid] = s.h[tid][tid];
  __syncthreads();
  sort_desc(s, rp);
  for (int e = tid; e < rp * k; e += SM_THREADS) {
    const int a = e / k, j = e - a * k;
    E[(long long)b * rp * k + e] = s.e[a][s.perm[j]];
  }
  if (tid < k) {
    const double lam = s.h[s.perm[tid]][s.perm[tid]];
    s.key[tid] = lam > 0.0 ? sqrt(lam) : 0.0;   // reuse: singular values
  }
  __syncthreads();
  if (tid == 0) {
    int ke = kcap;
    if (tau > 0.f) {
      const double thr = (double)tau * s.key[0];
      ke = 0;
      if (s.key[k - 1] < thr)
        for (int j = 0; j < k; ++j) ke += (s.key[j] > thr) ? 1 : 0;
      ke = ke < kcap ? ke : kcap;
    }
    keff[b] = ke;
    if (keff_user) keff_user[b] = ke;
    s.count = ke;
  }
  __syncthreads();
  const int ke = s.count;
  if (tid < k) {
    const double sj = s.key[tid];
    const float inv = sj > 0.0 ? (float)(1.0 / sj) : 0.f;
    sv[b * k + tid] = (float)sj;
    inv_sv[b * k + tid] = inv;
    coef_a[b * k + tid] = tid < ke ? -(float)sj : 0.f;
    if (s_user) s_user[b * k + tid] = (float)sj;
  }
}

// The head factors V = G^T E / s (k x s_pad, from the G^T panel Gt) and
// U = Q E (k x l_pad, from the Q panel Qt) of every matrix, from the float64
// eigenvectors E (rp x k, row-major) and the singular values of
// svd_head_kernel. One position per thread: the V positions, then the U
// positions, over ceil((s_pad + l_pad) / 256) work-groups per matrix, so both
// panels stream at full width. Each output sums its rp terms in row order in
// float64 and is rounded to float32 once (with E rounded to float32 first,
// the factors' columns lose orthogonality at float32 resolution, which the
// explicit restore's filter amplifies). V divides by the float32 singular
// value that the residual multiplies back. RM >= rp.
template <int RM>
__global__ __launch_bounds__(256) void head_factors_kernel(const double* __restrict__ E,
                                                           const float* __restrict__ sv, int rp, int k,
                                                           const float* __restrict__ Gt, long long sg, int s_pad,
                                                           const float* __restrict__ Qt, long long sq, int l_pad,
                                                           float* __restrict__ Vt, float* __restrict__ Ut) {
  __shared__ double es[RM * SM_MAX];
  __shared__ double isv[SM_MAX];
  const int per = (s_pad + l_pad + 255) / 256;
  const int b = blockIdx.x / per;
  const int x0 = (blockIdx.x - b * per) * 256 + threadIdx.x;
  const bool valid = x0 < s_pad + l_pad, vside = x0 < s_pad;
  const int x = !valid ? 0 : (vside ? x0 : x0 - s_pad);
  const float* P = vside ? Gt + b * sg : Qt + b * sq;
  const int ld = vside ? s_pad : l_pad;
  float v[RM];
#pragma unroll
  for (int r = 0; r < RM; ++r) v[r] = P[(long long)(r < rp ? r : rp - 1) * ld + x];
  for (int e = threadIdx.x; e < rp * k; e += 256) es[e] = E[(long long)b * rp * k + e];
  for (int j = threadIdx.x; j < k; j += 256) {
    const float sj = sv[b * k + j];
    isv[j] = sj > 0.f ? 1.0 / (double)sj : 0.0;
  }
  __syncthreads();
  if (!valid) return;
  float* out = (vside ? Vt + (long long)b * k * s_pad : Ut + (long long)b * k * l_pad) + x;
  for (int j = 0; j < k; ++j) {
    double acc = 0.0;
#pragma unroll
    for (int r = 0; r < RM; ++r)
      if (r < rp) acc = fma(es[r * k + j], (double)v[r], acc);
    out[(long long)j * ld] = (float)(vside ? isv[j] * acc : acc);
  }
}

// ------------------------------------------- Rayleigh-Ritz (Alg. 2) -------
// From the partials of T = V^T (Z V) (K x K, symmetrized): T = E diag(lam) E^T,
// Ritz pairs ordered by |lam| descending (ties: larger lam, then lower index).
// Deflated set I: all K (tau = 0) or the gate of Alg. 2 on the magnitudes.
// Coefficients for the residual (-lam), the padded start (sign(lam) / gamma)
// and the restore (max(lam, 0)). One work-group.
template <int NP>
__global__ __launch_bounds__(SM_THREADS) void ritz_kernel(const double* part, int nch, int K, float tau, int window,
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
  jacobi_eig_any<NP>(s, K);
  if (tid < K) s.key[tid] = fabs(s.h[tid][tid]);
  __syncthreads();
  if (tid < K) {
    const double k0 = order_key(s.key[tid]), lam = order_key(s.h[tid][tid]);
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const double kj = order_key(s.key[j]), lj = order_key(s.h[j][j]);
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
    s.count = nd;
  }
  __syncthreads();
  const int nd = s.count;
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
// j < kout, x < len (len a multiple of 128). scale may be null (1). Grid:
// (len / 128) * batch work-groups times RJ column groups of outputs
// (blockIdx.y: j = y, y + RJ, ...), so wide panels spread over more CUs;
// every global load of a thread is issued before its first use.
constexpr int ROT_RJ = 4;
template <int KM>
__global__ __launch_bounds__(128) void rotate_kernel(const float* __restrict__ in, long long si, int ldi,
                                                     const float* __restrict__ E, long long se,
                                                     const float* __restrict__ scale, long long ssc,
                                                     float* __restrict__ out, long long so, int ldo, int kin, int kout,
                                                     int len, int batch) {
  __shared__ float es[KM * KM];
  const int per = len / 128;
  const int b = blockIdx.x / per;
  const int x = (blockIdx.x - b * per) * 128 + threadIdx.x;
  constexpr int EL = KM * KM / 128;   // E entries per thread
  float ev[EL];
#pragma unroll
  for (int u = 0; u < EL; ++u) {
    const int e = threadIdx.x + 128 * u;
    ev[u] = e < kin * kout ? E[b * se + e] : 0.f;
  }
  float v[KM];
#pragma unroll
  for (int a = 0; a < KM; ++a) v[a] = a < kin ? in[b * si + (long long)a * ldi + x] : 0.f;
#pragma unroll
  for (int u = 0; u < EL; ++u) {
    const int e = threadIdx.x + 128 * u;
    if (e < kin * kout) es[e] = ev[u];
  }
  __syncthreads();
  for (int j = blockIdx.y; j < kout; j += ROT_RJ) {
    float acc = 0.f;
#pragma unroll
    for (int a = 0; a < KM; ++a)
      if (a < kin) acc += es[a * kout + j] * v[a];
    const float sc = scale ? scale[b * ssc + j] : 1.f;
    out[b * so + (long long)j * ldo + x] = sc * acc;
  }
}

}  // namespace sd
