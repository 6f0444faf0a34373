// Deflated polar factor ("msign") for batches of matrices: host orchestration
// and the C entry points. Pipeline per call (all on the caller's stream, no
// host synchronization):
//
//   canonical input X (s x l, s = min(m, n)); padded copy only if needed
//   Alg. 3:  Omega -> Y = X^T Omega -> CholQR -> J x (X Q, CholQR, X^T Y, CholQR)
//            -> G = (X Q)^T -> thin SVD via eig(G G^T) -> U = Q E, V = G^T E / s
//   Alg. 1:  nu = ||X - V S U^T||_F (residual pass), X0 = R / nu + U V^T / gamma
//   filter:  L steps of A = X X^T (symmetric tiles), B = b A + c A^2,
//            X <- a X + B X; the last step writes the caller's output.
#include "host.hpp"

namespace sd {

struct MsignPlan {
  int batch, m, n, k, steps, dtype;
  bool tall, copy_in;
  bool square;            // m == n: tall for Alg. 3 (A = M), filtered in place
  bool explicit_restore;  // head added after the filter (k > 0)
  int s, l, s_pad, l_pad, rp;
  int kw;                // estimated triplets: k, or the gate's window r when tau > 0 and window > 0
  int rq;                // rows of the sketch panels: rp rounded up to 32 (zero rows past rp)
  int rq16;              // rows of the split bf16 panel copies (hi, lo): 2 rp rounded up to 32
  size_t esz;
  // buffers
  void *xc, *bm;
  float *xa, *xb;        // float32 iterates (fp32 path)
  bf16_t *xa16, *xb16;   // bf16 path: the iterates as hi = bf16(X) (the product
  int8_t *xalo, *xblo;   // operand) plus e4m3 residual bytes
  float *a32;
  bf16_t* a16;
  double* E;             // leading eigenvectors of G G^T, [B][rp][kw] (float64)
  float *om, *yl, *ys, *sv, *invsv, *coefA, *coefB, *coefR, *coefG, *Ls, *Ll, *sumsq, *alpha, *nu;
  float* xl32;           // explicit restore, bf16 path: the filter output in float32
  bf16_t *om16, *yl16, *ys16;   // split bf16 copies of the panels: product operands (bf16 path)
  double *part, *fac;
  int* keff;
  int tiles;
};

static void plan_msign(MsignPlan& p, Arena& ar) {
  const size_t B = p.batch;
  const size_t sl = (size_t)p.s_pad * p.l_pad, ss = (size_t)p.s_pad * p.s_pad;
  p.xc = p.copy_in ? ar.take<char>(B * sl * p.esz) : nullptr;
  const bool bf = p.dtype == SD_DTYPE_BF16;
  p.xa = bf ? nullptr : ar.take<float>(B * sl);
  p.xb = bf ? nullptr : ar.take<float>(B * sl);
  p.xa16 = bf ? ar.take<bf16_t>(B * sl) : nullptr;
  p.xb16 = bf ? ar.take<bf16_t>(B * sl) : nullptr;
  p.xalo = bf ? ar.take<int8_t>(B * sl) : nullptr;
  p.xblo = bf ? ar.take<int8_t>(B * sl) : nullptr;
  p.a32 = ar.take<float>(B * ss);
  p.a16 = p.dtype == SD_DTYPE_BF16 ? ar.take<bf16_t>(B * ss) : nullptr;
  p.bm = ar.take<char>(B * ss * p.esz);
  const int kq = p.kw > 0 ? p.kw : 1;
  const int rq = p.rq, rq16 = p.rq16;
  p.om = ar.take<float>(B * rq * p.s_pad);
  p.yl = ar.take<float>(B * rq * p.l_pad);
  p.ys = ar.take<float>(B * rq * p.s_pad);
  p.om16 = bf ? ar.take<bf16_t>(B * rq16 * p.s_pad) : nullptr;
  p.yl16 = bf ? ar.take<bf16_t>(B * rq16 * p.l_pad) : nullptr;
  p.ys16 = bf ? ar.take<bf16_t>(B * rq16 * p.s_pad) : nullptr;
  p.E = ar.take<double>(B * rq * kq);
  p.sv = ar.take<float>(B * kq);
  p.invsv = ar.take<float>(B * kq);
  p.coefA = ar.take<float>(B * kq);
  p.coefB = ar.take<float>(B * kq);
  p.coefR = p.explicit_restore ? ar.take<float>(B * kq) : nullptr;
  p.coefG = bf ? nullptr : ar.take<float>(B * kq);
  p.xl32 = (p.explicit_restore && bf) ? ar.take<float>(B * sl) : nullptr;
  p.Ls = ar.take<float>(B * kq * p.s_pad);
  p.Ll = ar.take<float>(B * kq * p.l_pad);
  p.keff = ar.take<int>(B);
  p.part = ar.take<double>(gram_part_elems(p.batch, p.l_pad > p.s_pad ? p.l_pad : p.s_pad, rq, rq, true));
  p.fac = ar.take<double>(B * rq * rq);
  p.tiles = (p.s_pad / 128) * (p.l_pad / 128);
  p.sumsq = ar.take<float>(B * p.tiles);
  p.alpha = ar.take<float>(B);
  p.nu = ar.take<float>(B);
}

static int validate_msign(int batch, int m, int n, int k, int steps, int dtype, const void* in, const void* out,
                          const sd_msign_opts& o) {
  if (batch < 1 || m < 1 || n < 1 || k < 0 || steps < 0 || steps > 1000) return SD_ERR_INVALID_ARG;
  if (dtype != SD_DTYPE_F32 && dtype != SD_DTYPE_BF16) return SD_ERR_INVALID_ARG;
  if (!in || !out) return SD_ERR_INVALID_ARG;
  const int s = m < n ? m : n;
  if (k >= s) return SD_ERR_INVALID_ARG;
  if (o.oversample < 0 || o.power_iters < 0 || o.power_iters > 100) return SD_ERR_INVALID_ARG;
  if (!(o.gamma > 0.f) || !(o.tau >= 0.f) || !(o.tau < 1.f)) return SD_ERR_INVALID_ARG;
  if (o.restore != SD_RESTORE_PADDED && o.restore != SD_RESTORE_EXPLICIT) return SD_ERR_INVALID_ARG;
  if (o.window < 0 || o.window > s) return SD_ERR_INVALID_ARG;
  if (o.restore == SD_RESTORE_EXPLICIT && steps == 0) return SD_ERR_UNSUPPORTED;
  if ((long long)m * n > (1ll << 31) || (long long)batch * m * n > (1ll << 40)) return SD_ERR_UNSUPPORTED;
  if (k > 0) {
    const long long kw = (o.tau > 0.f && o.window > 0) ? o.window : k;
    const long long rp = kw + o.oversample < s ? kw + o.oversample : s;
    if (rp > SM_MAX) return SD_ERR_UNSUPPORTED;
  }
  return SD_OK;
}

static void make_plan(MsignPlan& p, int batch, int m, int n, int k, int steps, int dtype, const void* in,
                      const sd_msign_opts& o) {
  p.batch = batch;
  p.m = m;
  p.n = n;
  p.k = k;
  p.steps = steps;
  p.dtype = dtype;
  p.tall = m > n;
  p.square = m == n;
  p.s = p.tall ? n : m;
  p.l = p.tall ? m : n;
  p.s_pad = round_up(p.s, 128);
  p.l_pad = round_up(p.l, 128);
  p.kw = k > 0 ? ((o.tau > 0.f && o.window > 0) ? o.window : k) : 0;
  p.rp = k > 0 ? (p.kw + o.oversample < p.s ? p.kw + o.oversample : p.s) : 0;
  p.rq = p.rp > 32 ? 64 : 32;
  p.rq16 = split_rows(p.rp);
  p.esz = dtype == SD_DTYPE_BF16 ? 2 : 4;
  const bool aligned = in && (reinterpret_cast<uintptr_t>(in) % 16 == 0);
  p.copy_in = p.tall || p.s != p.s_pad || p.l != p.l_pad || !aligned;
  p.explicit_restore = o.restore == SD_RESTORE_EXPLICIT && k > 0;
}

// Iterate update X <- a X + B X on 128 x 128 tiles; the epilogue's X reads
// are issued before the main loop. bf16 path: operand tiles move into a
// two-stage LDS ring by direct-to-LDS loads, two work-groups per CU; fp32
// path: register-staged tiles.
template <typename T, typename SX, typename Epi>
static void update_gemm(const MsignPlan& p, const T* bm, const SX* xop, const GemmShape& g, const Epi& eu,
                        hipStream_t st) {
  (void)p;
  if constexpr (sizeof(T) == 2) launch_gemm_dma<CfgDma128, true, false>(bm, xop, g, eu, st);
  else launch_gemm<CfgTile128, T, true, false>(bm, xop, g, eu, st);
}

// Symmetric products (Gram and A^2) on 128 x 128 tiles, upper-triangle tiles
// only; direct-to-LDS loads on the bf16 path.
template <typename T, typename Epi>
static void sym_gemm(const T* a, const GemmShape& g, const Epi& e, hipStream_t st) {
  if constexpr (sizeof(T) == 2) launch_gemm_dma<CfgDma128, false, true>(a, a, g, e, st);
  else launch_gemm<CfgTile128, T, false, true>(a, a, g, e, st);
}

// Residual floor rho of the padded start, relative to ||X||_F: the rounding
// level of the float32 arithmetic that forms the residual on both paths (the
// bf16 path's sketch products take split panels, so its head is float32-
// class too). R = X - V S U^T is a float32 difference of X and a rank-k
// float32 product whose entries are as large as X's, built from head factors
// that carry float32 rounding, so its rounding is a few units of 2^-24
// ||X||_F; a residual within rho = 16 u = 2^-20 of ||X||_F is that rounding
// (the input has rank <= k_eff, outside Alg. 1's k < rank(M)) and is dropped.
constexpr float kResidualFloor = 0x1p-20f;

template <typename T>
static int run_msign(const MsignPlan& p, const float* coeffs, const sd_msign_opts& o, const T* in, T* out,
                     hipStream_t st) {
  const int B = p.batch;
  const long long sl = (long long)p.s_pad * p.l_pad, ss = (long long)p.s_pad * p.s_pad;
  // canonical input
  const T* xc;
  long long sx;
  int ldx;
  if (p.copy_in) {
    T* dst = reinterpret_cast<T*>(p.xc);
    const int blocks = (p.s_pad / 32) * (p.l_pad / 32) * B;
    hipLaunchKernelGGL((canon_copy_kernel<T>), dim3(blocks), dim3(256), 0, st, dst, sl, p.l_pad, p.s_pad,
                       p.l_pad, in, (long long)p.m * p.n, p.s, p.l, p.tall ? 1 : 0, B);
    xc = dst;
    sx = sl;
    ldx = p.l_pad;
  } else {
    xc = in;
    sx = (long long)p.m * p.n;
    ldx = p.l;
  }

  // Alg. 3: head estimate. Panels are [B][rq][len_pad] (rows past rp zero);
  // on the bf16 path the products take the panels' bf16 copies and run on
  // the direct-to-LDS GEMM.
  if (p.k > 0) {
    const int rp = p.rp, rq = p.rq, s_pad = p.s_pad, l_pad = p.l_pad;
    const long long so = (long long)rq * s_pad, sl_ = (long long)rq * l_pad;
    constexpr bool BF = sizeof(T) == 2;
    // the sketch kernels write the whole padded panels (zero rows past rp,
    // zero columns past s); the CholQR passes write the bf16 copies of Q
    // likewise, so no panel needs clearing first
    const int rq16 = p.rq16, nrow = BF && rq16 > rq ? rq16 : rq;
    const long long so16 = (long long)rq16 * s_pad;
    if (o.sketch) {
      const long long tot = (long long)nrow * s_pad * B;
      hipLaunchKernelGGL(sketch_copy_kernel, grid1(tot, 256), dim3(256), 0, st, p.om, so, s_pad, o.sketch, p.s, rp, rq,
                         B, BF ? p.om16 : nullptr, so16, rq16);
    } else {
      const long long tot = (long long)nrow * (s_pad / 4) * B;
      hipLaunchKernelGGL(sketch_kernel, grid1(tot, 256), dim3(256), 0, st, p.om, so, s_pad, p.s, rp, rq, o.seed, B,
                         BF ? p.om16 : nullptr, so16, rq16);
    }
    // bf16 path: split-panel products (float32-class results); fp32 path:
    // fp64 accumulation
    auto xtw = [&](const float* w, const bf16_t* w16, float* out) {
      if constexpr (BF)
        ts_xtw_dma(reinterpret_cast<const bf16_t*>(xc), sx, ldx, s_pad, l_pad, w16, rq16, rp, out, rq, B, st);
      else ts_xtw<T, true>(xc, sx, ldx, s_pad, l_pad, w, so, s_pad, rp, out, sl_, l_pad, B, st);
    };
    auto xw = [&](const float* w, const bf16_t* w16, float* out) {
      if constexpr (BF)
        ts_xw_dma(reinterpret_cast<const bf16_t*>(xc), sx, ldx, s_pad, l_pad, w16, rq16, rp, out, rq, B, st);
      else ts_xw<T, true>(xc, sx, ldx, s_pad, l_pad, w, sl_, l_pad, rp, out, so, s_pad, B, st);
    };
    // Alg. 3 takes A = M for n >= m: the sketch multiplies the columns of the
    // tall orientation. A wide input (X = M) and a tall one (X = M^T after the
    // canonical copy) both have A = X^T, so Omega multiplies X's rows: Y
    // lives on the l side, G = Q^T A on the s side. A square input is tall
    // (A = M = X) and is sketched from the other side without a copy: Y = X
    // Omega on the s side, G^T = X^T Q on the l side, and the head factors
    // change sides (U = Q E on the rows of X, V = G^T E / s on its columns).
    // The Gram, polynomial and update of the filter are the same either way.
    const bool sq = p.square;
    float* pq = sq ? p.ys : p.yl;   // Q and Y (the sketched side)
    float* pg = sq ? p.yl : p.ys;   // the other side: power-iteration panel, then G^T
    bf16_t* pq16 = sq ? p.ys16 : p.yl16;
    bf16_t* pg16 = sq ? p.yl16 : p.ys16;
    const long long sq_ = sq ? so : sl_, sg_ = sq ? sl_ : so;
    const int lq = sq ? s_pad : l_pad, lg = sq ? l_pad : s_pad;
    auto to_q = [&](const float* w, const bf16_t* w16, float* out) {   // product onto the sketched side
      if (sq) xw(w, w16, out);
      else xtw(w, w16, out);
    };
    auto to_g = [&](const float* w, const bf16_t* w16, float* out) {   // product onto the other side
      if (sq) xtw(w, w16, out);
      else xw(w, w16, out);
    };
    to_q(p.om, p.om16, pq);
    cholqr(pq, sq_, lq, rp, lq, B, p.part, p.fac, o.status_dev, st, pq16, rq16);
    for (int j = 0; j < o.power_iters; ++j) {
      to_g(pq, pq16, pg);
      cholqr(pg, sg_, lg, rp, lg, B, p.part, p.fac, o.status_dev, st, pg16, rq16);
      to_q(pg, pg16, pq);
      cholqr(pq, sq_, lq, rp, lq, B, p.part, p.fac, o.status_dev, st, pq16, rq16);
    }
    to_g(pq, pq16, pg);   // G^T = A^T Q
    {
      ProfScope ps(SD_STAGE_SMALL, st);
      gram_partials(pg, sg_, lg, pg, sg_, lg, rp, rp, lg, true, p.part, B, st);   // G G^T
#define SD_HEAD(NPV)                                                                                       \
  hipLaunchKernelGGL(svd_head_kernel<NPV>, dim3(B), dim3(SM_THREADS), 0, st, p.part, lg / GP_CHUNK, rp, p.kw, \
                     p.k, o.tau, p.E, p.sv, p.invsv, p.keff, p.coefA, o.s_out, o.k_eff_out)
      switch (jacobi_class(rp)) {
        case 4: SD_HEAD(4); break;
        case 8: SD_HEAD(8); break;
        case 12: SD_HEAD(12); break;
        case 16: SD_HEAD(16); break;
        case 32: SD_HEAD(32); break;
        default: SD_HEAD(0); break;
      }
#undef SD_HEAD
      // V = G^T E / s onto the G side's factor, U = Q E onto the Q side's
      // (Ls: the rows of X, Ll: its columns; s_pad = l_pad when square)
      float* vt = sq ? p.Ll : p.Ls;
      float* ut = sq ? p.Ls : p.Ll;
      const dim3 gf(((s_pad + l_pad + 255) / 256) * B);
      if (rp <= 16)
        hipLaunchKernelGGL(head_factors_kernel<16>, gf, dim3(256), 0, st, p.E, p.sv, rp, p.kw, pg, sg_, lg, pq,
                           sq_, lq, vt, ut);
      else if (rp <= 32)
        hipLaunchKernelGGL(head_factors_kernel<32>, gf, dim3(256), 0, st, p.E, p.sv, rp, p.kw, pg, sg_, lg, pq,
                           sq_, lq, vt, ut);
      else
        hipLaunchKernelGGL(head_factors_kernel<SM_MAX>, gf, dim3(256), 0, st, p.E, p.sv, rp, p.kw, pg, sg_, lg,
                           pq, sq_, lq, vt, ut);
    }
  } else if (o.k_eff_out) {
    hipLaunchKernelGGL(fill_int_kernel, grid1(B, 256), dim3(256), 0, st, o.k_eff_out, (long long)B, 0);
  }

  // Alg. 1: residual norm and padded start
  LowRankArgs la{};
  la.x = xc;
  la.sx = sx;
  la.ldx = ldx;
  la.L = p.Ls;   // V = G^T E / s, [kw][s_pad]
  la.sl = (long long)p.kw * p.s_pad;
  la.ldl = p.s_pad;
  la.Rr = p.Ll;  // U = Q E, [kw][l_pad]
  la.sr = (long long)p.kw * p.l_pad;
  la.ldr = p.l_pad;
  la.kk = p.k > 0 ? p.keff : nullptr;
  la.kconst = 0;
  la.kmax = p.kw > 0 ? p.kw : 1;
  la.rows_pad = p.s_pad;
  la.cols_pad = p.l_pad;
  la.batch = B;
  la.coef = p.coefA;
  la.coef2 = nullptr;
  la.alpha = nullptr;
  la.out = nullptr;
  la.sumsq = p.sumsq;
  // fp32 path: R = X - V S U^T formed in float64 (two-term start below)
  constexpr bool R64 = sizeof(T) == 4;
  lowrank<T, T, R64>(la, st);
  {
    ProfScope ps(SD_STAGE_LOWRANK, st);
    hipLaunchKernelGGL(muon_finalize_kernel, dim3(B), dim3(64), 0, st, p.sumsq, p.tiles, p.sv,
                       p.k > 0 ? p.keff : nullptr, la.kmax, p.explicit_restore ? 0.f : 1.f / o.gamma,
                       kResidualFloor, p.alpha, p.coefB, p.nu, o.nu_out, p.coefR, p.coefG, o.status_dev, B);
  }
  // X0 = alpha R + gamma^-1 V U^T: fp32 path as alpha (X - V S U^T) + V (1 / gamma) U^T
  // (coefA, coefG); bf16 path in one term, alpha X + V (-(s alpha - 1 / gamma)) U^T (coefB)
  la.coef = R64 ? p.coefA : p.coefB;
  la.coef2 = R64 ? p.coefG : nullptr;
  la.alpha = p.alpha;
  la.out = p.xa;        // fp32 path: float32 X0
  la.out16 = p.xa16;    // bf16 path: X0 as hi plus 8-bit residuals
  la.out_lo = p.xalo;
  la.so = sl;
  la.ldo = p.l_pad;
  la.sumsq = nullptr;
  lowrank<T, float, R64>(la, st);

  // fixed-depth filter: float32 iterate (fp32 path) or hi = bf16(X) plus
  // e4m3 residual bytes, hi being the product operand (bf16 path)
  float* cur = p.xa;
  float* nxt = p.xb;
  bf16_t* cur16 = p.xa16;
  bf16_t* nxt16 = p.xb16;
  int8_t* curlo = p.xalo;
  int8_t* nxtlo = p.xblo;
  T* bm = reinterpret_cast<T*>(p.bm);
  constexpr bool BF = sizeof(T) == 2;
  auto xop = [&]() -> const T* {
    if constexpr (BF) return reinterpret_cast<const T*>(cur16);
    else return reinterpret_cast<const T*>(cur);
  };
  for (int t = 0; t < p.steps; ++t) {
    const float a = coeffs ? coeffs[3 * t] : 3.4445f;
    const float b = coeffs ? coeffs[3 * t + 1] : -4.7750f;
    const float c = coeffs ? coeffs[3 * t + 2] : 2.0315f;
    GemmShape g1{p.s_pad, p.s_pad, p.l_pad, p.l_pad, p.l_pad, sl, sl, B};
    EpiGram eg{};
    eg.stride = ss;
    eg.ld = p.s_pad;
    if (c != 0.f) {
      eg.out32 = p.a32;
      eg.scale32 = 1.f;
      eg.out16 = BF ? p.a16 : nullptr;
      eg.scale16 = 1.f;
    } else if (BF) {
      eg.out16 = reinterpret_cast<bf16_t*>(bm);
      eg.scale16 = b;
    } else {
      eg.out32 = reinterpret_cast<float*>(bm);
      eg.scale32 = b;
    }
    // bf16 path: the Gram's copies and B stay cacheable for their reader
    // when small enough (stream_outputs)
    {
      ProfScope ps(SD_STAGE_NS_GRAM, st);
      if constexpr (BF) {
        if (stream_outputs((long long)B * ss * ((eg.out32 ? 4 : 0) + (eg.out16 ? 2 : 0))))
          sym_gemm<T>(xop(), g1, eg, st);
        else
          sym_gemm<T>(xop(), g1, cached_stores(eg), st);
      } else {
        sym_gemm<T>(xop(), g1, eg, st);
      }
    }
    if (c != 0.f) {
      GemmShape g2{p.s_pad, p.s_pad, p.s_pad, p.s_pad, p.s_pad, ss, ss, B};
      EpiPoly<T> ep{p.a32, bm, b, c, ss, p.s_pad};
      const T* aop = BF ? reinterpret_cast<const T*>(p.a16) : reinterpret_cast<const T*>(p.a32);
      ProfScope ps(SD_STAGE_NS_POLY, st);
      if constexpr (BF) {
        if (stream_outputs((long long)B * ss * 2)) sym_gemm<T>(aop, g2, ep, st);
        else sym_gemm<T>(aop, g2, cached_stores(ep), st);
      } else {
        sym_gemm<T>(aop, g2, ep, st);
      }
    }
    GemmShape g3{p.s_pad, p.l_pad, p.s_pad, p.s_pad, p.l_pad, ss, sl, B, 1};
    const bool last = t + 1 == p.steps;
    ProfScope ps(SD_STAGE_NS_UPDATE, st);
    if constexpr (BF) {
      if (last && p.explicit_restore) {
        // the filter output stays float32 (canonical layout) for the restore
        EpiUpdateHL<float> ef{};
        ef.hi = cur16;
        ef.lo = curlo;
        ef.xstride = sl;
        ef.ldx = p.l_pad;
        ef.ac = a;
        ef.out = p.xl32;
        ef.ostride = sl;
        ef.ldo = p.l_pad;
        ef.final_out = 1;
        ef.transpose_out = 0;
        ef.rows_valid = p.s_pad;
        ef.cols_valid = p.l_pad;
        update_gemm<T>(p, bm, xop(), g3, ef, st);
        continue;
      }
      EpiUpdateHL<T> eu{};
      eu.hi = cur16;
      eu.lo = curlo;
      eu.xstride = sl;
      eu.ldx = p.l_pad;
      eu.ac = a;
      if (!last) {
        eu.out_hi = nxt16;
        eu.out_lo = nxtlo;
        eu.final_out = 0;
      } else {
        eu.out = out;
        eu.ostride = (long long)p.m * p.n;
        eu.ldo = p.tall ? p.s : p.l;
        eu.final_out = 1;
        eu.transpose_out = p.tall ? 1 : 0;
        eu.rows_valid = p.s;
        eu.cols_valid = p.l;
      }
      update_gemm<T>(p, bm, xop(), g3, eu, st);
    } else if (!last || p.explicit_restore) {
      EpiUpdate<float, float> eu{};
      eu.x = cur;
      eu.xstride = sl;
      eu.ldx = p.l_pad;
      eu.ac = a;
      eu.out = nxt;
      eu.ostride = sl;
      eu.ldo = p.l_pad;
      eu.final_out = 0;
      update_gemm<T>(p, bm, xop(), g3, eu, st);
    } else {
      EpiUpdate<float, T> eu{};
      eu.x = cur;
      eu.xstride = sl;
      eu.ldx = p.l_pad;
      eu.ac = a;
      eu.out = out;
      eu.ostride = (long long)p.m * p.n;
      eu.ldo = p.tall ? p.s : p.l;
      eu.final_out = 1;
      eu.transpose_out = p.tall ? 1 : 0;
      eu.rows_valid = p.s;
      eu.cols_valid = p.l;
      update_gemm<T>(p, bm, xop(), g3, eu, st);
    }
    float* tmp = cur;
    cur = nxt;
    nxt = tmp;
    bf16_t* tmp16 = cur16;
    cur16 = nxt16;
    nxt16 = tmp16;
    int8_t* tmplo = curlo;
    curlo = nxtlo;
    nxtlo = tmplo;
  }
  if (p.explicit_restore) {
    // out = X_L + U_k V_k^T (eq:identities), rounded once to the output type:
    // straight into the caller's buffer when its layout is the canonical one,
    // else through the canonical input buffer (free after the front end)
    LowRankArgs ra = la;
    if constexpr (BF) ra.x = p.xl32;
    else ra.x = cur;   // the last update's target (the buffers were swapped after it)
    ra.sx = sl;
    ra.ldx = p.l_pad;
    ra.coef = p.coefR;
    ra.coef2 = nullptr;
    ra.alpha = nullptr;
    ra.out16 = nullptr;
    ra.out_lo = nullptr;
    ra.sumsq = nullptr;
    const bool direct = !p.copy_in && reinterpret_cast<uintptr_t>(out) % 16 == 0;
    ra.out = direct ? static_cast<void*>(out) : p.xc;
    ra.so = direct ? (long long)p.m * p.n : sl;
    ra.ldo = direct ? p.l : p.l_pad;
    lowrank<float, T>(ra, st);
    if (!direct) {
      const long long tot = (long long)p.m * p.n * B;
      hipLaunchKernelGGL((store_out_kernel<T, T>), grid1(tot, 256), dim3(256), 0, st, reinterpret_cast<const T*>(p.xc),
                         sl, p.l_pad, out, (long long)p.m * p.n, p.s, p.l, p.tall ? 1 : 0, B);
    }
  }
  if (p.steps == 0) {
    // the start itself, rounded to the output type (bf16 path: its hi)
    const long long tot = (long long)p.m * p.n * B;
    if constexpr (BF)
      hipLaunchKernelGGL((store_out_kernel<bf16_t, T>), grid1(tot, 256), dim3(256), 0, st, cur16, sl, p.l_pad, out,
                         (long long)p.m * p.n, p.s, p.l, p.tall ? 1 : 0, B);
    else
      hipLaunchKernelGGL((store_out_kernel<float, T>), grid1(tot, 256), dim3(256), 0, st, cur, sl, p.l_pad, out,
                         (long long)p.m * p.n, p.s, p.l, p.tall ? 1 : 0, B);
  }
  return hip_status();
}

static int msign_enqueue(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                         const void* in, void* out, const sd_msign_opts& o, hipStream_t stream);

}  // namespace sd

using namespace sd;

extern "C" {

void sd_msign_opts_default(sd_msign_opts* o) {
  if (!o) return;
  *o = sd_msign_opts{};
  o->oversample = 8;
  o->power_iters = 1;
  o->gamma = 1.01f;
  o->tau = 0.f;
  o->seed = 0;
}

size_t sd_msign_workspace_bytes(int batch, int m, int n, int k, int dtype, const sd_msign_opts* opts) {
  sd_msign_opts o;
  sd_msign_opts_default(&o);
  if (opts) o = *opts;
  const char dummy[16] __attribute__((aligned(16))) = {0};
  if (validate_msign(batch, m, n, k, 1, dtype, dummy, dummy, o) != SD_OK) return 0;
  MsignPlan p{};
  // assume the input needs a copy (upper bound over alignments)
  make_plan(p, batch, m, n, k, 0, dtype, nullptr, o);
  Arena ar;
  plan_msign(p, ar);
  return ar.off + 256;
}

int sd_msign_deflated_ex(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                         const void* in, void* out, const sd_msign_opts* opts, hipStream_t stream) {
  sd_msign_opts o;
  sd_msign_opts_default(&o);
  if (opts) o = *opts;
  int rc = validate_msign(batch, m, n, k, steps, dtype, in, out, o);
  if (rc != SD_OK) return rc;
  return sd::msign_enqueue(batch, m, n, k, steps, coeffs, dtype, in, out, o, stream);
}
}  // extern "C"

namespace sd {
// Enqueue one validated call.
static int msign_enqueue(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                         const void* in, void* out, const sd_msign_opts& o, hipStream_t stream) {
  int rc;
  MsignPlan p{};
  make_plan(p, batch, m, n, k, steps, dtype, in, o);
  Arena sizing;
  plan_msign(p, sizing);
  Scratch scratch;
  rc = scratch.acquire(o.workspace, o.workspace_bytes, sizing.off + 256, stream);
  if (rc != SD_OK) return rc;
  Arena ar;
  ar.base = reinterpret_cast<char*>(scratch.ptr);
  plan_msign(p, ar);
  if (dtype == SD_DTYPE_BF16)
    rc = run_msign<bf16_t>(p, coeffs, o, reinterpret_cast<const bf16_t*>(in), reinterpret_cast<bf16_t*>(out),
                           stream);
  else
    rc = run_msign<float>(p, coeffs, o, reinterpret_cast<const float*>(in), reinterpret_cast<float*>(out), stream);
  scratch.release();
  return rc;
}

// Library-owned streams for concurrent groups: per device, created on first
// use (non-blocking, default priority) and kept until the process ends, with
// one fork event and one join event per stream.
struct GroupStreams {
  static constexpr int N = 3;
  hipStream_t s[N] = {};
  hipEvent_t fork = nullptr, join[N] = {};
  bool ready = false;
};

static int group_streams(GroupStreams*& gs) {
  static std::mutex mu;
  static GroupStreams per_dev[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return SD_ERR_HIP;
  std::lock_guard<std::mutex> g(mu);
  GroupStreams& d = per_dev[dev];
  if (!d.ready) {
    for (int i = 0; i < GroupStreams::N; ++i) {
      if (hipStreamCreateWithFlags(&d.s[i], hipStreamNonBlocking) != hipSuccess) return SD_ERR_HIP;
      if (hipEventCreateWithFlags(&d.join[i], hipEventDisableTiming) != hipSuccess) return SD_ERR_HIP;
    }
    if (hipEventCreateWithFlags(&d.fork, hipEventDisableTiming) != hipSuccess) return SD_ERR_HIP;
    d.ready = true;
  }
  gs = &d;
  return SD_OK;
}
// one host thread at a time enqueues on the shared group streams and events
static std::mutex group_enqueue_mu;

// ------------------------------------------- parameter-list grouping -----
// Gather (staging is the destination, s x l row-major per member) or scatter
// (staging is the source) for up to PL_MAX members per launch; a member whose
// own layout is l x s (tall) is transposed through a 32 x 32 LDS tile so
// that both its reads and its writes are coalesced. Grid: (cdiv(s, 32) *
// cdiv(l, 32), members); 256 threads.
constexpr int PL_MAX = 32;
struct ParamTable {
  const void* src[PL_MAX];
  void* dst[PL_MAX];
  int transpose[PL_MAX];
};

template <typename T>
__global__ __launch_bounds__(256) void param_copy_kernel(ParamTable t, int s, int l, int gather) {
  __shared__ T tile[32][33];
  const int b = blockIdx.y;
  const int tl = (l + 31) / 32;
  const int i0 = (blockIdx.x / tl) * 32, j0 = (blockIdx.x % tl) * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const T* src = reinterpret_cast<const T*>(t.src[b]);
  T* dst = reinterpret_cast<T*>(t.dst[b]);
  if (!t.transpose[b]) {   // both sides s x l
    for (int r = ty; r < 32; r += 8) {
      const int i = i0 + r, j = j0 + tx;
      if (i < s && j < l) dst[(long long)i * l + j] = src[(long long)i * l + j];
    }
    return;
  }
  if (gather) {   // src l x s: staging[i][j] = src[j][i]
    for (int r = ty; r < 32; r += 8) {
      const int j = j0 + r, i = i0 + tx;
      tile[r][tx] = (j < l && i < s) ? src[(long long)j * s + i] : T{};
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
      const int i = i0 + r, j = j0 + tx;
      if (i < s && j < l) dst[(long long)i * l + j] = tile[tx][r];
    }
  } else {        // dst l x s: dst[j][i] = staging[i][j]
    for (int r = ty; r < 32; r += 8) {
      const int i = i0 + r, j = j0 + tx;
      tile[r][tx] = (i < s && j < l) ? src[(long long)i * l + j] : T{};
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
      const int j = j0 + r, i = i0 + tx;
      if (j < l && i < s) dst[(long long)j * s + i] = tile[tx][r];
    }
  }
}

// Gather or scatter one group's members (param indices `idx`) against the
// staging batch `stg` (s x l per member, esz bytes per element).
static void param_copy(const sd_msign_param* params, const std::vector<int>& idx, char* stg, int s, int l,
                       size_t esz, bool gather, hipStream_t st) {
  const size_t per = (size_t)s * l * esz;
  const dim3 blk(256);
  for (size_t c0 = 0; c0 < idx.size(); c0 += PL_MAX) {
    ParamTable t{};
    const int nb = (int)std::min<size_t>(PL_MAX, idx.size() - c0);
    for (int u = 0; u < nb; ++u) {
      const sd_msign_param& q = params[idx[c0 + u]];
      char* mine = stg + (c0 + u) * per;
      t.src[u] = gather ? q.in : mine;
      t.dst[u] = gather ? static_cast<void*>(mine) : q.out;
      t.transpose[u] = q.m > q.n;
    }
    const dim3 grid((unsigned)(cdiv(s, 32) * cdiv(l, 32)), (unsigned)nb);
    if (esz == 2) hipLaunchKernelGGL(param_copy_kernel<uint16_t>, grid, blk, 0, st, t, s, l, gather ? 1 : 0);
    else hipLaunchKernelGGL(param_copy_kernel<float>, grid, blk, 0, st, t, s, l, gather ? 1 : 0);
  }
}
}  // namespace sd

extern "C" {

int sd_msign_groups(int ngroups, const sd_msign_group* groups, hipStream_t stream) {
  if (ngroups < 1 || !groups) return SD_ERR_INVALID_ARG;
  std::vector<sd_msign_opts> opts(ngroups);
  for (int i = 0; i < ngroups; ++i) {
    const sd_msign_group& g = groups[i];
    sd_msign_opts_default(&opts[i]);
    if (g.opts) opts[i] = *g.opts;
    const int rc = validate_msign(g.batch, g.m, g.n, g.k, g.steps, g.dtype, g.in, g.out, opts[i]);
    if (rc != SD_OK) return rc;
  }
  if (ngroups == 1) {
    const sd_msign_group& g = groups[0];
    return msign_enqueue(g.batch, g.m, g.n, g.k, g.steps, g.coeffs, g.dtype, g.in, g.out, opts[0], stream);
  }
  GroupStreams* gs = nullptr;
  int rc = group_streams(gs);
  if (rc != SD_OK) return rc;
  std::lock_guard<std::mutex> lock(group_enqueue_mu);
  const int used = ngroups < GroupStreams::N ? ngroups : GroupStreams::N;
  if (hipEventRecord(gs->fork, stream) != hipSuccess) return SD_ERR_HIP;
  for (int i = 0; i < used; ++i)
    if (hipStreamWaitEvent(gs->s[i], gs->fork, 0) != hipSuccess) return SD_ERR_HIP;
  for (int i = 0; i < ngroups && rc == SD_OK; ++i) {
    const sd_msign_group& g = groups[i];
    rc = msign_enqueue(g.batch, g.m, g.n, g.k, g.steps, g.coeffs, g.dtype, g.in, g.out, opts[i],
                       gs->s[i % GroupStreams::N]);
  }
  // join every used stream back, also after a failure, so `stream` never runs ahead
  for (int i = 0; i < used; ++i) {
    if (hipEventRecord(gs->join[i], gs->s[i]) != hipSuccess || hipStreamWaitEvent(stream, gs->join[i], 0) != hipSuccess)
      return SD_ERR_HIP;
  }
  return rc;
}

int sd_msign_params(int count, const sd_msign_param* params, int k, int steps, const float* coeffs, int dtype,
                    const sd_msign_opts* opts, hipStream_t stream) {
  if (count < 1 || !params) return SD_ERR_INVALID_ARG;
  sd_msign_opts o;
  sd_msign_opts_default(&o);
  if (opts) o = *opts;
  if (o.workspace) return SD_ERR_INVALID_ARG;
  // buckets by (s, l) in order of first appearance, members in list order
  std::vector<std::pair<int, int>> keys;
  std::vector<std::vector<int>> members;
  for (int i = 0; i < count; ++i) {
    const sd_msign_param& q = params[i];
    if (!q.in || !q.out || q.m < 1 || q.n < 1) return SD_ERR_INVALID_ARG;
    const std::pair<int, int> key(std::min(q.m, q.n), std::max(q.m, q.n));
    size_t g = 0;
    while (g < keys.size() && keys[g] != key) ++g;
    if (g == keys.size()) {
      keys.push_back(key);
      members.emplace_back();
    }
    members[g].push_back(i);
  }
  const char probe[16] __attribute__((aligned(16))) = {0};
  for (size_t g = 0; g < keys.size(); ++g) {
    const int rc = validate_msign((int)members[g].size(), keys[g].first, keys[g].second, k, steps, dtype, probe,
                                  probe, o);
    if (rc != SD_OK) return rc;
  }
  const size_t esz = dtype == SD_DTYPE_BF16 ? 2 : 4;
  GroupStreams* gs = nullptr;
  int rc = group_streams(gs);
  if (rc != SD_OK) return rc;
  std::lock_guard<std::mutex> lock(group_enqueue_mu);
  const int used = (int)std::min<size_t>(keys.size(), GroupStreams::N);
  if (hipEventRecord(gs->fork, stream) != hipSuccess) return SD_ERR_HIP;
  for (int i = 0; i < used; ++i)
    if (hipStreamWaitEvent(gs->s[i], gs->fork, 0) != hipSuccess) return SD_ERR_HIP;
  for (size_t g = 0; g < keys.size() && rc == SD_OK; ++g) {
    hipStream_t st = gs->s[g % GroupStreams::N];
    const int s = keys[g].first, l = keys[g].second, b = (int)members[g].size();
    const size_t bytes = (size_t)b * s * l * esz, half = (bytes + 255) / 256 * 256;
    Scratch stg;
    rc = stg.acquire(nullptr, 0, 2 * half, st);
    if (rc != SD_OK) break;
    char* in = reinterpret_cast<char*>(stg.ptr);
    char* out = in + half;
    param_copy(params, members[g], in, s, l, esz, true, st);
    rc = msign_enqueue(b, s, l, k, steps, coeffs, dtype, in, out, o, st);
    if (rc == SD_OK) param_copy(params, members[g], out, s, l, esz, false, st);
    stg.release();
  }
  // join every used stream back, also after a failure, so `stream` never runs ahead
  for (int i = 0; i < used; ++i) {
    if (hipEventRecord(gs->join[i], gs->s[i]) != hipSuccess || hipStreamWaitEvent(stream, gs->join[i], 0) != hipSuccess)
      return SD_ERR_HIP;
  }
  if (rc == SD_OK) rc = hip_status();
  return rc;
}

int sd_sketch(int batch, int s, int rp, uint64_t seed, float* out, hipStream_t stream) {
  if (batch < 1 || s < 1 || rp < 1 || !out) return SD_ERR_INVALID_ARG;
  const long long tot = (long long)rp * ((s + 3) / 4) * batch;
  hipLaunchKernelGGL(sketch_kernel, grid1(tot, 256), dim3(256), 0, stream, out, (long long)s * rp, s, s, rp, rp, seed,
                     batch, (bf16_t*)nullptr, 0ll, 0);
  return hip_status();
}

int sd_sketch_host(int batch, int s, int rp, uint64_t seed, float* out) {
  if (batch < 1 || s < 1 || rp < 1 || !out) return SD_ERR_INVALID_ARG;
  const long long per = (long long)s * rp;
  for (int b = 0; b < batch; ++b)
    for (long long call = 0; call < (per + 3) / 4; ++call) {
      float z[4];
      Philox::normals(z, (uint32_t)call, (uint32_t)b, 1u, seed);
      for (int t = 0; t < 4; ++t) {
        const long long g = 4 * call + t;
        if (g < per) out[(long long)b * per + g] = z[t];
      }
    }
  return SD_OK;
}

}  // extern "C"

namespace sd {
// Scratch of the allocation-free entry point: one array per device, held
// until the process ends. Host code never passes its name to a kernel (in
// host code the name stands for a host-side shadow): each device's address
// comes from hipGetSymbolAddress, taken once per device with that device
// current, and only that address is used.
constexpr size_t kStaticScratchBytes = (size_t)SD_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

static int static_scratch(void** ptr) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return SD_ERR_HIP;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) {
      (void)hipGetLastError();
      return SD_ERR_HIP;
    }
    addr[dev] = a;
  }
  *ptr = addr[dev];
  return SD_OK;
}
}  // namespace sd

extern "C" {

int sd_msign_deflated_noalloc(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                              const void* in, void* out, const sd_msign_opts* opts, hipStream_t stream) {
  sd_msign_opts o;
  sd_msign_opts_default(&o);
  if (opts) o = *opts;
  if (o.workspace) return SD_ERR_INVALID_ARG;   // the scratch is the library's
  int rc = validate_msign(batch, m, n, k, steps, dtype, in, out, o);
  if (rc != SD_OK) return rc;
  // the call's scratch (the input's alignment decides only whether the
  // canonical copy is needed, so the query with a copy is an upper bound)
  const size_t need = sd_msign_workspace_bytes(batch, m, n, k, dtype, &o);
  if (need == 0 || need > kStaticScratchBytes) return SD_ERR_WORKSPACE;
  void* ws = nullptr;
  rc = static_scratch(&ws);
  if (rc != SD_OK) return rc;
  o.workspace = ws;
  o.workspace_bytes = kStaticScratchBytes;
  return sd::msign_enqueue(batch, m, n, k, steps, coeffs, dtype, in, out, o, stream);
}

int sd_msign(int batch, int m, int n, int steps, const float* coeffs, const float* in, float* out,
             hipStream_t stream) {
  return sd_msign_deflated_ex(batch, m, n, 0, steps, coeffs, SD_DTYPE_F32, in, out, nullptr, stream);
}
int sd_msign_deflated(int batch, int m, int n, int k, int steps, const float* coeffs, const float* in,
                      float* out, hipStream_t stream) {
  return sd_msign_deflated_ex(batch, m, n, k, steps, coeffs, SD_DTYPE_F32, in, out, nullptr, stream);
}
int sd_msign_bf16(int batch, int m, int n, int steps, const float* coeffs, const uint16_t* in, uint16_t* out,
                  hipStream_t stream) {
  return sd_msign_deflated_ex(batch, m, n, 0, steps, coeffs, SD_DTYPE_BF16, in, out, nullptr, stream);
}
int sd_msign_deflated_bf16(int batch, int m, int n, int k, int steps, const float* coeffs, const uint16_t* in,
                           uint16_t* out, hipStream_t stream) {
  return sd_msign_deflated_ex(batch, m, n, k, steps, coeffs, SD_DTYPE_BF16, in, out, nullptr, stream);
}

}  // extern "C"
