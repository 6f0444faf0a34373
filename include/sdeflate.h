/*
 * sdeflate: spectrally deflated fixed-depth polynomial matrix filters on
 * AMD Instinct MI355X (gfx950).
 *
 * Method: "Spectral Deflation for Factorization-Free Matrix Filtering in Muon
 * and Semidefinite Programming" (arXiv 2609.21102). A fixed-depth polynomial
 * filter X_t = p_t(X_{t-1}) started from a normalized input (eq:filter) is
 * run on the residual left after removing an estimated dominant rank-k part;
 * the removed part is padded back into the start (Muon) or restored after the
 * filter (PSD projection). Deflation leaves the target matrix function
 * unchanged (eq:identities).
 *
 * Conventions shared by every entry point
 *   - Data pointers are DEVICE pointers owned by the caller. Matrices are
 *     dense, row-major and contiguous. Coefficient tables are HOST pointers,
 *     read before the call returns.
 *   - Work is enqueued on `stream` (0 = the null stream) and never waits for
 *     the device; results are ready when the stream reaches that point.
 *   - Return value: SD_OK, or a negative sd_status. Argument errors are
 *     reported synchronously and nothing is enqueued. SD_ERR_HIP reports a
 *     failed allocation or launch. Numerical events found on the device are
 *     reported through the optional `status_dev` word of the options.
 *   - Non-finite input (NaN, Inf) is not checked: it propagates to the output
 *     of the matrix that holds it (other matrices of a batch are unaffected),
 *     and the call completes; every index the kernels derive from values
 *     (orderings of singular and Ritz values, deflation counts) stays in range.
 *   - Without a caller workspace the library allocates one per call from the
 *     device's stream-ordered memory pool (hipMallocAsync / hipFreeAsync on
 *     `stream`), so calls on different streams do not share scratch memory.
 *   - `in` may equal `out`: the input is fully consumed before the output is
 *     written.
 *   - Random numbers (the Gaussian sketch of Alg. 3, the Lanczos start vector)
 *     come from Philox4x32-10 with key = seed and counter = (call, matrix,
 *     stream, 0) and a float64 Box-Muller transform; identical seeds give
 *     identical results, run to run.
 */
#ifndef SDEFLATE_H
#define SDEFLATE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SD_OK = 0,
  SD_ERR_INVALID_ARG = -1, /* bad sizes, null pointers, options out of range */
  SD_ERR_UNSUPPORTED = -2, /* valid but not supported (e.g. sketch wider than 64) */
  SD_ERR_HIP = -3,         /* HIP allocation or launch failure */
  SD_ERR_NUMERIC = -4,     /* reserved: numerical failures are flagged in status_dev */
  SD_ERR_WORKSPACE = -5    /* caller workspace smaller than the *_workspace_bytes query */
} sd_status;

enum { SD_DTYPE_F32 = 0, SD_DTYPE_BF16 = 1 };

/* Bits set (atomically OR-ed) in *status_dev when the device meets them. */
enum {
  SD_FLAG_PIVOT_FLOOR = 2,   /* a CholeskyQR pivot hit its floor: a rank-deficient panel */
  SD_FLAG_RESIDUAL_FLOOR = 4 /* Muon: a residual at the float32 rounding level of the head
                                was dropped (nu <= 2^-20 ||X||_F: the input has rank
                                <= k_eff, outside Alg. 1's k < rank(M)); X0 is then
                                gamma^-1 U_k V_k^T (0 with the explicit restore) */,
  SD_FLAG_EIG_UNCONVERGED = 8 /* PSD, tracked bases wider than 32: the block Jacobi
                                Rayleigh-Ritz reached its cap of 16 sweeps with the
                                off-diagonal mass above 2^-40 of the norm */
};

/* ------------------------------------------------------------------ Muon --
 * Deflated polar factor, batched (Alg. 1 with the batched randomized SVD of
 * Alg. 3). For every matrix M of the batch [batch, m, n]:
 *   - orientation: a matrix with m > n is processed as M^T and its result
 *     transposed back, polar(M^T) = polar(M)^T (App. D, grouping);
 *   - head estimate: Alg. 3 with r' = min(min(m, n), r + oversample) sketch
 *     columns (r = k, or the gate's window when set) and power_iters subspace
 *     iterations, one CholeskyQR pass after every product (float64 Gram and
 *     factorization), thin SVD of the r' x min(m,n) reduced matrix;
 *   - deflation rank: k (fixed rank, tau = 0), or the gate of Alg. 1 on the
 *     r estimated values: if s_r < tau s_1 deflate min(k, max{i : s_i >
 *     tau s_1}) components, else none;
 *   - start: X0 = R / ||R||_F + gamma^-1 U_k V_k^T with R = M - U_k S_k V_k^T
 *     (Alg. 1), or X0 = M / ||M||_F when nothing is deflated; a zero norm
 *     drops its term, so a zero matrix maps to zero;
 *   - filter: L = steps steps X <- a_t X + (b_t A + c_t A^2) X with A the Gram
 *     of the short side (eq:muon_ns; Polar-Express-style tables give one row
 *     per step).
 * coeffs: HOST float[steps][3] (a_t, b_t, c_t), or NULL for Muon's retuned
 *   quintic (3.4445, -4.7750, 2.0315) at every step (Sec. 3 setup).
 * Precision: the f32 entry points compute in float32 (MFMA fp32, float32
 *   accumulation); their sketch products accumulate in float64 and the
 *   residual M - U_k S_k V_k^T is formed in float64 (rounded once). The bf16
 *   entry points take bfloat16 input and output (uint16_t bit patterns). Their
 *   front end runs at float32 precision: the sketch products take each float32
 *   panel as two bf16 operands (hi, lo) with float32 accumulation. Every
 *   product of the filter takes bf16 operands with float32 accumulation. The
 *   iterate is stored in 3 bytes per element: hi = bf16(X), the product
 *   operand, plus an OCP float8 e4m3 byte holding (X - hi) 2^16, carried as
 *   hi + e4m3 2^-16. The Gram A is kept in float32 (rounded to bf16 where it
 *   is a product operand), b A + c A^2 is rounded to bf16, and the sketch
 *   panels, norms and small factorizations are float32 / float64.
 * Requirements: batch >= 1, m, n >= 1, 0 <= k < min(m, n), k + oversample
 *   capped at min(m, n) must not exceed 64 (else SD_ERR_UNSUPPORTED),
 *   0 <= steps <= 1000. k = 0 is the undeflated baseline, and the gated
 *   variant that deflates nothing returns the baseline bit for bit (Sec. 2.2).
 * Orientation of the sketch: Alg. 3 takes A = M for n >= m (square included)
 *   and A = M^T for a wide M, and sketches A's columns (Y = A Omega).
 */
/* How the deflated head returns (eq:identities: polar(M) = U_k V_k^T + polar(R_k)):
 *   PADDED (Alg. 1): X0 = R / ||R||_F + gamma^-1 U_k V_k^T, and the filter
 *     itself drives the head toward 1;
 *   EXPLICIT (the gamma -> infinity form): X0 = R / ||R||_F, and U_k V_k^T is
 *     added to the filter's output (in float32, before the final rounding).
 *     gamma is unused. Needs steps >= 1 (SD_ERR_UNSUPPORTED otherwise). */
enum { SD_RESTORE_PADDED = 0, SD_RESTORE_EXPLICIT = 1 };

typedef struct {
  int oversample;          /* p >= 0, default 8 */
  int power_iters;         /* J >= 0, default 1 */
  float gamma;             /* padding, > 0, default 1.01 */
  float tau;               /* 0 = fixed rank k (default); in (0, 1): gate of Alg. 1 */
  uint64_t seed;           /* Philox key, default 0 */
  const float* sketch;     /* optional device [batch][r'][min(m,n)]: Omega column j of
                              matrix b at sketch + (b * r' + j) * min(m,n); NULL = Philox */
  void* workspace;         /* optional device scratch, >= sd_msign_workspace_bytes() */
  size_t workspace_bytes;
  int* k_eff_out;          /* optional device int[batch]: deflated components */
  float* nu_out;           /* optional device float[batch]: norm X0 was scaled by */
  float* s_out;            /* optional device float[batch][r]: estimated singular values
                              (r = window when the gate's window is set, else k) */
  int* status_dev;         /* optional device int: SD_FLAG_* bits are OR-ed in */
  int restore;             /* SD_RESTORE_PADDED (default) or SD_RESTORE_EXPLICIT */
  int window;              /* gate window r of Alg. 1, used only with tau > 0: 0 (default) = k;
                              else 1 <= r <= min(m, n): r values are estimated (r' = min(min(m,n),
                              r + oversample)) and the gate deflates min(k, max{i : s_i > tau s_1})
                              of them when s_r < tau s_1 */
} sd_msign_opts;

void sd_msign_opts_default(sd_msign_opts* opts);

int sd_msign(int batch, int m, int n, int steps, const float* coeffs, const float* in, float* out,
             hipStream_t stream);
int sd_msign_deflated(int batch, int m, int n, int k, int steps, const float* coeffs, const float* in,
                      float* out, hipStream_t stream);
int sd_msign_bf16(int batch, int m, int n, int steps, const float* coeffs, const uint16_t* in,
                  uint16_t* out, hipStream_t stream);
int sd_msign_deflated_bf16(int batch, int m, int n, int k, int steps, const float* coeffs,
                           const uint16_t* in, uint16_t* out, hipStream_t stream);
/* dtype: SD_DTYPE_F32 or SD_DTYPE_BF16 for both in and out; opts may be NULL. */
int sd_msign_deflated_ex(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                         const void* in, void* out, const sd_msign_opts* opts, hipStream_t stream);
/* One shape group of a Muon step: the arguments of one sd_msign_deflated_ex
 * call (opts may be NULL; a workspace in opts serves that group alone). */
typedef struct {
  int batch, m, n, k, steps;
  const float* coeffs;        /* HOST [steps][3] or NULL */
  int dtype;                  /* SD_DTYPE_F32 or SD_DTYPE_BF16 */
  const void* in;
  void* out;
  const sd_msign_opts* opts;
} sd_msign_group;

/* The deflated polar factors of a whole Muon step: a parameter list grouped
 * by shape, one batched call per group (App. D, "Grouping"; here the
 * grouping itself, wide vs tall and equal shapes, is the caller's:
 * sd_msign_params below does it in the library). Every group is
 * validated first: on an argument error nothing is enqueued and the error of
 * the first bad group is returned. The groups then run concurrently on
 * library-owned streams (default priority, at most three per device) that
 * wait for `stream` and are joined back into it, so the results are ready
 * when `stream` reaches that point, as with one call. Each group's result is
 * the one sd_msign_deflated_ex gives for it alone, bit for bit. Scratch comes
 * from the pool on the group's stream unless its opts bring a workspace.
 * The output buffers of different groups must not overlap. */
int sd_msign_groups(int ngroups, const sd_msign_group* groups, hipStream_t stream);

/* One matrix of a Muon step's parameter list: in and out are m x n row-major
 * of the call's dtype, device memory; out may equal in (updated in place)
 * but may not otherwise overlap any other parameter's in or out. */
typedef struct sd_msign_param {
  const void* in;
  void* out;
  int m, n;
} sd_msign_param;

/* The deflated polar factors of a parameter list with the grouping done by
 * the library (App. D, "Grouping"): parameters are bucketed by shape with
 * wide ones transposed (polar(M^T) = polar(M)^T), so an m x n and an n x m
 * matrix share the group of s x l, s = min(m, n), l = max(m, n); groups are
 * formed in order of first appearance in the list, and a group's batch holds
 * its members in list order (member b is matrix b of that batch: its sketch
 * is Philox matrix b of the call). Each group is gathered into one s x l batch
 * (tall members transposed), runs as one batched sd_msign_deflated_ex call
 * with k, steps, coeffs, dtype and opts, and is scattered back (transposed
 * back where it was gathered transposed); groups run concurrently as in
 * sd_msign_groups, joined back into `stream`. Every parameter's result is
 * bit for bit the one of that batched call. All parameters are validated
 * first (SD_ERR_INVALID_ARG: count < 1, a null pointer, m or n < 1,
 * k >= min(m, n), or invalid opts; nothing is enqueued then). Staging
 * buffers (two per group, batch x s x l elements) and each group's scratch
 * come from the pool on the group's stream; opts->workspace must be NULL.
 * A pool allocation that fails (SD_ERR_HIP) stops the enqueueing there: the
 * groups enqueued before it still run and are joined into `stream`. */
int sd_msign_params(int count, const sd_msign_param* params, int k, int steps, const float* coeffs, int dtype,
                    const sd_msign_opts* opts, hipStream_t stream);

/* Workspace an _ex call with these arguments needs (0 on invalid arguments). */
size_t sd_msign_workspace_bytes(int batch, int m, int n, int k, int dtype, const sd_msign_opts* opts);

/* Allocation-free form of sd_msign_deflated_ex, for callers that cannot
 * allocate device memory during the call (code captured into a HIP graph,
 * serving loops, harnesses that forbid hipMalloc): same arguments, results
 * and errors, but its scratch is a library-owned array of
 * SD_STATIC_SCRATCH_BYTES per GPU (a static device array, held until the
 * process ends), and it calls no hipMalloc / hipFree or allocating routine.
 * Calls whose sd_msign_workspace_bytes() exceeds that size return
 * SD_ERR_WORKSPACE with nothing enqueued (at bf16 that is one 768 x 3072
 * matrix, or about 24 of 768 x 768); opts->workspace must be NULL
 * (SD_ERR_INVALID_ARG otherwise). Every call on one GPU shares the array and
 * overwrites it: calls that overlap on one GPU (other streams, other host
 * threads) race and must be ordered by the caller. No part of the scratch
 * needs to start at zero. */
#define SD_STATIC_SCRATCH_BYTES (64u << 20)
int sd_msign_deflated_noalloc(int batch, int m, int n, int k, int steps, const float* coeffs, int dtype,
                              const void* in, void* out, const sd_msign_opts* opts, hipStream_t stream);
/* The Gaussian sketch Alg. 3 draws (Omega ~ N(0, 1)^{s x r'} per matrix): out[b][j][i]
 * is entry (i, j) of matrix b's sketch, Gaussian number j * s + i of Philox stream 1.
 * sd_sketch fills a DEVICE buffer on `stream`; sd_sketch_host computes the same
 * numbers on the host into a HOST buffer (batch * rp * s floats). */
int sd_sketch(int batch, int s, int rp, uint64_t seed, float* out, hipStream_t stream);
int sd_sketch_host(int batch, int s, int rp, uint64_t seed, float* out);

/* ------------------------------------------------------------------- PSD --
 * Deflated projection onto the PSD cone of a symmetric X (n x n, float32),
 * one projection of Alg. 2:
 *   - (subspace_iters - 1) pre-steps V <- CholeskyQR(X V) on the basis V =
 *     Qwarm (n x k, orthonormal columns, row-major);
 *   - Zt = X V; Rayleigh-Ritz on V^T Zt; Ritz pairs ordered by |lambda|
 *     descending (ties: larger lambda, then lower index);
 *   - deflated set: all k pairs (tau = 0), or the gate of Alg. 2 with window
 *     r: if s_r < tau s_1, the pairs with |lambda| > tau s_1, else none;
 *   - R = X - sum lambda u u^T; theta = Lanczos upper estimate of ||R||_2
 *     (App. E.1: lanczos_steps steps on R^2, largest Ritz pair (rho, v),
 *     theta = sqrt(rho + ||R^2 v - rho v||)); X0 = R / theta + gamma^-1
 *     sum sign(lambda) u u^T;
 *   - g = steps steps of the odd polynomial filter X <- a X + (b A + c A^2) X,
 *     A = X^2 (cubic: c = 0; default (a, b) = (3/2, -1/2), the d = 1
 *     Newton-Schulz map of eq:general_ns_iteration);
 *   - P = R (I + g) / 2 + sum_{lambda > 0} lambda u u^T, then (P + P^T) / 2;
 *     with nothing deflated, P = X (I + g(X / theta)) / 2 symmetrized
 *     (eq:baseline_projection);
 *   - Qwarm <- CholeskyQR(Zt) (the basis for the next call).
 * Everything is float32 (MFMA fp32), small factorizations float64.
 * Tracked bases up to 32 columns keep their K x K problems in one
 * work-group's LDS; wider ones (up to 512, the paper's K = ceil(0.05 n) at
 * its SDP sizes) take float64 panel products, a one-work-group Cholesky
 * with a block-row solve, a block Jacobi Rayleigh-Ritz and float32 MFMA
 * GEMMs for the rank-K terms, and compute the next basis on a
 * library-owned side stream (default priority) joined back into `stream`.
 * Requirements: n >= 1, 0 <= k < n, k <= 512, 0 <= steps <= 1000; Qwarm is
 * required when k > 0 and must not overlap X or out. k = 0 is the baseline
 * (Qwarm unused, may be NULL).
 */
/* Arithmetic of the sign filter's products (the paper's SDP experiments run
 * the filter in fp16, App. E): SD_PREC_F32 computes them in float32 (fp32
 * MFMA); SD_PREC_F16 rounds every product operand to fp16 (round to nearest
 * even) and accumulates in float32 (fp16 MFMA), the restore product R g
 * included, whose operands are fp16(R / theta) and fp16(g) (scaled back by
 * theta). The iterate, the Gram and b A + c A^2 are stored in float32 either
 * way, and the residual, the Ritz step and the Lanczos scale stay float32. */
enum { SD_PREC_F32 = 0, SD_PREC_F16 = 1 };

/* Normalization scale theta of the residual (X0 = R / theta + ...):
 * SD_SCALE_LANCZOS (default): the Lanczos upper estimate of ||R||_2 of
 *   App. E.1 (lanczos_steps steps on R^2 from the seeded start);
 * SD_SCALE_FROBENIUS: theta = ||R||_F (>= ||R||_2, no iteration), the residual
 *   Frobenius-normalized as Alg. 1 normalizes the Muon residual; it lowers the
 *   floor of X0's spectrum by up to sqrt(n) against the Lanczos scale. */
enum { SD_SCALE_LANCZOS = 0, SD_SCALE_FROBENIUS = 1 };

typedef struct {
  int subspace_iters;      /* J >= 1, default 1 */
  int lanczos_steps;       /* 1..64, default 20 */
  float gamma;             /* padding, > 0, default 1.1 */
  float tau;               /* 0 = deflate all k Ritz pairs (default); in (0, 1): gate */
  int window;              /* r of the gate, 1..k (used when tau > 0) */
  int poly_degree;         /* 3 (default) or 5 */
  const float* poly;       /* HOST float[steps][(poly_degree + 1) / 2] or NULL = (1.5, -0.5) */
  uint64_t seed;           /* Philox key of the Lanczos start, default 0 */
  void* workspace;
  size_t workspace_bytes;
  int* n_deflated_out;     /* optional device int */
  int* n_positive_out;     /* optional device int */
  float* theta_out;        /* optional device float */
  float* ritz_out;         /* optional device float[k], Ritz values in deflation order */
  int* status_dev;         /* optional device int */
  int precision;           /* SD_PREC_F32 (default) or SD_PREC_F16, see below */
  int scale_mode;          /* SD_SCALE_LANCZOS (default) or SD_SCALE_FROBENIUS, see below */
} sd_psd_opts;

void sd_psd_opts_default(sd_psd_opts* opts);

int sd_psd_project(int n, int steps, const float* X, float* out, hipStream_t stream);
int sd_psd_project_deflated(int n, int k, int steps, const float* X, float* Qwarm, float* out,
                            hipStream_t stream);
int sd_psd_project_deflated_ex(int n, int k, int steps, const float* X, float* Qwarm, float* out,
                               const sd_psd_opts* opts, hipStream_t stream);
size_t sd_psd_workspace_bytes(int n, int k, const sd_psd_opts* opts);

/* ------------------------------------------------------------------ ADMM --
 * Three-block ADMM (App. E.1, eq:admm_iter) for the standard-form SDP pair
 * with diagonal constraints, min <C, X> s.t. diag(X) = b, X PSD (the max-cut
 * relaxation; A X = diag(X), A* y = Diag(y), A A* = I, so the y-update is
 * elementwise), penalty sigma > 0, for `iters` iterations:
 *     y = b / sigma - diag(X / sigma + S - C),   Z = C - Diag(y) - X / sigma,
 *     S = projection of Z,                       X = X + sigma (S + Diag(y) - C).
 * The projection is sd_psd_project_deflated_ex with `opts` (filter steps,
 * gamma, gate tau / window, precision, ...) on the tracked basis Qwarm
 * [n, k] (in/out: one block step and CholQR per iteration, Alg. 2), with the
 * gate held closed for the first `warmup` iterations while the basis settles
 * (Sec. 3.3); k = 0 projects with the undeflated baseline.
 * C, b: device [n, n] (symmetric) and [n]. X, S [n, n] and y [n]: device,
 * in/out (the iteration continues from them; zeros start it afresh).
 * eta_out: optional device float[iters], the eigenvalue-free KKT residual
 * after each iteration (the first three terms of eq:admm_eta). ndef_out:
 * optional device int[iters], the deflated count of each projection.
 * The per-projection outputs of opts (n_deflated_out, n_positive_out,
 * theta_out, ritz_out) are not used. Scratch: opts->workspace of
 * sd_admm_workspace_bytes(), or the pool. The caller owns every buffer;
 * the call is asynchronous on `stream`. Errors, returned with nothing
 * enqueued: SD_ERR_INVALID_ARG for n < 1, iters < 0, warmup < 0, sigma <= 0,
 * steps outside 0..1000,
 * a null C, b, X, S or y, k < 0 or k >= n, k > 0 without Qwarm, a basis
 * overlapping C or S, or invalid opts; SD_ERR_UNSUPPORTED for k > 512.
 * iters = 0 validates and returns SD_OK. */
int sd_admm_diag(int n, int iters, int steps, float sigma, const float* C, const float* b, float* X, float* S,
                 float* y, int k, float* Qwarm, int warmup, const sd_psd_opts* opts, float* eta_out, int* ndef_out,
                 hipStream_t stream);
size_t sd_admm_workspace_bytes(int n, int k, int steps, const sd_psd_opts* opts);

/* ---------------------------------------------------------- stage timing --
 * Benchmark instrumentation (tracing). While a stage's bit (1 << stage) is set
 * in the mask, the library brackets every launch of that stage with a pair of
 * HIP events recorded on the call's stream; this adds two event records per
 * launch and nothing else. sd_profile_read waits for the recorded events
 * (a host synchronization), adds their elapsed times to the running totals
 * and returns the totals of one stage. sd_profile_reset clears the totals.
 * The instrumentation state is process-wide.
 */
enum {
  SD_STAGE_NS_GRAM = 0,    /* A = X X^T (symmetric tiles) */
  SD_STAGE_NS_POLY = 1,    /* B = b A + c A^2 */
  SD_STAGE_NS_UPDATE = 2,  /* X <- a X + B X */
  SD_STAGE_SKETCH = 3,     /* tall-skinny products of Alg. 3 / the subspace step */
  SD_STAGE_CHOLQR = 4,     /* CholeskyQR of the panels */
  SD_STAGE_SMALL = 5,      /* small SVD / Rayleigh-Ritz / rotations */
  SD_STAGE_LOWRANK = 6,    /* residual norm, padded start, PSD residual */
  SD_STAGE_LANCZOS = 7,    /* Lanczos scale estimate */
  SD_STAGE_RESTORE = 8,    /* PSD restore product and symmetrized output */
  SD_STAGE_COUNT = 9
};
void sd_profile_set(unsigned mask);
int sd_profile_read(int stage, double* total_ms, long long* launches);
void sd_profile_reset(void);

/* ---------------------------------------------------------------- misc ---- */
const char* sd_status_string(int status);
int sd_version(void); /* major * 10000 + minor * 100 + patch */

#ifdef __cplusplus
}
#endif

#endif /* SDEFLATE_H */
