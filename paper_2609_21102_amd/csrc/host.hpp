// Host-side helpers: workspace carving, stream-ordered scratch allocation and
// kernel dispatch by compile-time widths.
#pragma once

#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "../../include/sdeflate.h"
#include "common.hpp"
#include "gemm.hpp"
#include "lowrank.hpp"
#include "skinny.hpp"
#include "small.hpp"

namespace sd {

// Bump allocator over one block; with base == nullptr it only measures.
struct Arena {
  char* base = nullptr;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// Scratch for one call: the caller's workspace, or a block from the device's
// stream-ordered pool (released on the same stream at the end of the call).
struct Scratch {
  void* ptr = nullptr;
  bool owned = false;
  hipStream_t stream = nullptr;
  int acquire(void* user, size_t user_bytes, size_t need, hipStream_t st) {
    stream = st;
    if (user) {
      if (user_bytes < need) return SD_ERR_WORKSPACE;
      ptr = user;
      return SD_OK;
    }
    if (need == 0) return SD_OK;
    static std::once_flag once[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return SD_ERR_HIP;
    if (dev >= 0 && dev < 64)
      std::call_once(once[dev], [dev]() {
        hipMemPool_t pool;
        if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
          uint64_t keep = ~0ull;   // keep freed blocks cached in the pool
          (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
        }
      });
    if (hipMallocAsync(&ptr, need, st) != hipSuccess) {
      ptr = nullptr;
      (void)hipGetLastError();
      return SD_ERR_HIP;
    }
    owned = true;
    return SD_OK;
  }
  void release() {
    if (owned && ptr) (void)hipFreeAsync(ptr, stream);
    ptr = nullptr;
    owned = false;
  }
  ~Scratch() { release(); }
};

// ------------------------------------------------------ stage timing ------
// When a stage's bit is set (sd_profile_set), every launch of that stage is
// bracketed by two HIP events on the call's stream. sd_profile_read waits for
// the recorded events and accumulates their elapsed times per stage.
struct Profiler {
  std::mutex mu;
  unsigned mask = 0;
  struct Rec {
    int stage;
    hipEvent_t a, b;
  };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  double total_ms[SD_STAGE_COUNT] = {};
  long long launches[SD_STAGE_COUNT] = {};
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  void drain() {
    for (auto& r : pending) {
      float ms = 0.f;
      if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
        total_ms[r.stage] += ms;
        launches[r.stage] += 1;
      }
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    pending.clear();
  }
};
inline Profiler& profiler() {
  static Profiler p;
  return p;
}
struct ProfScope {
  int stage;
  hipStream_t st;
  hipEvent_t a = nullptr;
  ProfScope(int s, hipStream_t stream) : stage(s), st(stream) {
    Profiler& p = profiler();
    if (!(p.mask & (1u << s))) return;
    std::lock_guard<std::mutex> g(p.mu);
    a = p.get();
    if (a) (void)hipEventRecord(a, st);
  }
  ~ProfScope() {
    if (!a) return;
    Profiler& p = profiler();
    std::lock_guard<std::mutex> g(p.mu);
    hipEvent_t b = p.get();
    if (!b) return;
    (void)hipEventRecord(b, st);
    p.pending.push_back({stage, a, b});
  }
};

inline int hip_status() { return hipGetLastError() == hipSuccess ? SD_OK : SD_ERR_HIP; }

inline dim3 grid1(long long n, int block) { return dim3((unsigned)((n + block - 1) / block)); }

inline void fill(float* p, long long n, float v, hipStream_t st) {
  if (n > 0) hipLaunchKernelGGL(fill_kernel, grid1(n, 256), dim3(256), 0, st, p, n, v);
}

// ----------------------------------------------------------- dispatch -----
template <typename T, bool ACC64 = false>
void ts_xtw(const T* X, long long sx, int ldx, int s_pad, int l_pad, const float* Wt, long long sw, int ldw,
            int rp, float* Pt, long long sp, int ldp, int batch, hipStream_t st) {
  ProfScope ps(SD_STAGE_SKETCH, st);
  const dim3 g((l_pad / 128) * batch), b(256);
  switch (cdiv(rp, 16)) {
    case 1: hipLaunchKernelGGL((ts_xtw_kernel<T, 1, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    case 2: hipLaunchKernelGGL((ts_xtw_kernel<T, 2, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    case 3: hipLaunchKernelGGL((ts_xtw_kernel<T, 3, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    default: hipLaunchKernelGGL((ts_xtw_kernel<T, 4, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
  }
}

template <typename T, bool ACC64 = false>
void ts_xw(const T* X, long long sx, int ldx, int s_pad, int l_pad, const float* Wt, long long sw, int ldw,
           int rp, float* Pt, long long sp, int ldp, int batch, hipStream_t st) {
  ProfScope ps(SD_STAGE_SKETCH, st);
  const dim3 g((s_pad / 16) * batch), b(256);
  switch (cdiv(rp, 16)) {
    case 1: hipLaunchKernelGGL((ts_xw_kernel<T, 1, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    case 2: hipLaunchKernelGGL((ts_xw_kernel<T, 2, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    case 3: hipLaunchKernelGGL((ts_xw_kernel<T, 3, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
    default: hipLaunchKernelGGL((ts_xw_kernel<T, 4, ACC64>), g, b, 0, st, X, sx, ldx, s_pad, l_pad, Wt, sw, ldw, rp, Pt, sp, ldp, batch); break;
  }
}

// bf16 tall-skinny products on the direct-to-LDS GEMM. The operand panel W16
// holds each of the rp panel rows split in two bf16 rows, hi = bf16(w) in row
// j and lo = bf16(w - hi) in row rp + j (zero rows up to rq16), so that with
// the exact bf16 X the product of a float32 panel is formed to about 2^-17 of
// its value instead of bf16's 2^-9; the epilogue adds each row pair. Results
// are fp32 panels Pt [batch][rq][len_pad] (rows rp .. rq - 1 written as zero).
//   ts_xtw_dma:  Pt = (X^T W)^T = W^T X       (M = rq16, N = l_pad, K = s_pad, X in NN form)
//   ts_xw_dma:   Pt = (X W)^T   = W^T X^T     (M = rq16, N = s_pad, K = l_pad, X rows in NT form)
inline void ts_xtw_dma(const bf16_t* X, long long sx, int ldx, int s_pad, int l_pad, const bf16_t* W16, int rq16,
                       int rp, float* Pt, int rq, int batch, hipStream_t st) {
  ProfScope ps(SD_STAGE_SKETCH, st);
  GemmShape g{rq16, l_pad, s_pad, s_pad, ldx, (long long)rq16 * s_pad, sx, batch};
  EpiStoreRowsSplit e{Pt, (long long)rq * l_pad, l_pad, rp, rq};
  if (rq16 == 32) launch_gemm_dma<GemmCfg<1, 4, 1, 1, 2, 0>, true, false>(W16, X, g, e, st);
  else if (rq16 == 64) launch_gemm_dma<GemmCfg<1, 4, 2, 1, 2, 0>, true, false>(W16, X, g, e, st);
  else launch_gemm_dma<GemmCfg<1, 4, 4, 1, 2, 0>, true, false>(W16, X, g, e, st);
}
inline void ts_xw_dma(const bf16_t* X, long long sx, int ldx, int s_pad, int l_pad, const bf16_t* W16, int rq16,
                      int rp, float* Pt, int rq, int batch, hipStream_t st) {
  ProfScope ps(SD_STAGE_SKETCH, st);
  GemmShape g{rq16, s_pad, l_pad, l_pad, ldx, (long long)rq16 * l_pad, sx, batch};
  EpiStoreRowsSplit e{Pt, (long long)rq * s_pad, s_pad, rp, rq};
  // one wave per 32-column tile and a four-stage ring: the K loop is long
  // (l_pad) and the grid small, so more loads per work-group stay in flight
  if (rq16 == 32) launch_gemm_dma<GemmCfg<1, 1, 1, 1, 4, 0>, false, false>(W16, X, g, e, st);
  else if (rq16 == 64) launch_gemm_dma<GemmCfg<1, 1, 2, 1, 4, 0>, false, false>(W16, X, g, e, st);
  else launch_gemm_dma<GemmCfg<1, 1, 4, 1, 4, 0>, false, false>(W16, X, g, e, st);
}

// Rows of the split bf16 operand copy of a panel with rp rows.
inline int split_rows(int rp) { return 2 * rp <= 32 ? 32 : (2 * rp <= 64 ? 64 : 128); }

// Float64 partial Grams of panel rows over 128-position chunks.
inline void gram_partials(const float* A, long long sa, int lda, const float* B, long long sb, int ldb, int ca,
                          int cb, int len_pad, bool sym, double* part, int batch, hipStream_t st) {
  const dim3 g((len_pad / GP_CHUNK) * batch), b(256);
  const int cm = ca > cb ? ca : cb;
  if (cm > 16 && sym && A == B && sa == sb && lda == ldb && ca == cb) {
    // one panel of more than 16 rows: the blocked kernel (at 16 rows and
    // fewer its one-entry blocks measured slower than the kernel below)
    if (cm <= 32) hipLaunchKernelGGL((gram_partial_sym_kernel<32, 2>), g, b, 0, st, A, sa, lda, ca, len_pad, part, batch);
    else hipLaunchKernelGGL((gram_partial_sym_kernel<64, 4>), g, b, 0, st, A, sa, lda, ca, len_pad, part, batch);
    return;
  }
  if (cm <= 16) hipLaunchKernelGGL((gram_partial_kernel<16>), g, b, 0, st, A, sa, lda, B, sb, ldb, ca, cb, len_pad, sym, part, batch);
  else if (cm <= 32) hipLaunchKernelGGL((gram_partial_kernel<32>), g, b, 0, st, A, sa, lda, B, sb, ldb, ca, cb, len_pad, sym, part, batch);
  else hipLaunchKernelGGL((gram_partial_kernel<64>), g, b, 0, st, A, sa, lda, B, sb, ldb, ca, cb, len_pad, sym, part, batch);
}

// Scratch of the panel factorizations: partial Grams and the factors.
inline size_t gram_part_elems(int batch, int len_pad, int ca, int cb, bool sym) {
  return (size_t)batch * (len_pad / GP_CHUNK) * gram_items(ca, cb, sym);
}

// One CholeskyQR pass on every panel of the batch, in place (plus, with Pt16,
// the split bf16 copy of Q: hi rows 0 .. c - 1, lo rows c .. 2c - 1, zero
// rows up to c16; [batch][c16][ld]).
inline void cholqr(float* Pt, long long sp, int ld, int c, int len_pad, int batch, double* part, double* fac,
                   int* status, hipStream_t st, bf16_t* Pt16 = nullptr, int c16 = 0) {
  const long long sp16 = (long long)c16 * ld;
  ProfScope ps(SD_STAGE_CHOLQR, st);
  gram_partials(Pt, sp, ld, Pt, sp, ld, c, c, len_pad, true, part, batch, st);
  const int nch = len_pad / GP_CHUNK;
  const dim3 g((len_pad / 128) * batch), b(128);
  if (c <= 16) {
    hipLaunchKernelGGL((chol_qr_kernel<16>), g, b, 0, st, Pt, sp, ld, c, len_pad, part, nch, status, Pt16, c16, sp16);
  } else {   // wider panels: factor on one work-group per panel, then apply
    hipLaunchKernelGGL(chol_factor_kernel, dim3(batch), dim3(256), 0, st, part, nch, c, fac, status);
    if (c <= 32) hipLaunchKernelGGL((chol_apply_kernel<32>), g, b, 0, st, Pt, sp, ld, c, len_pad, fac, batch, Pt16, c16, sp16);
    else hipLaunchKernelGGL((chol_apply_kernel<64>), g, b, 0, st, Pt, sp, ld, c, len_pad, fac, batch, Pt16, c16, sp16);
  }
}

inline void rotate(const float* in, long long si, int ldi, const float* E, long long se, const float* scale,
                   long long ssc, float* out, long long so, int ldo, int kin, int kout, int len, int batch,
                   hipStream_t st) {
  ProfScope ps(SD_STAGE_SMALL, st);
  const dim3 g((len / 128) * batch, ROT_RJ), b(128);
  if (kin <= 16) hipLaunchKernelGGL((rotate_kernel<16>), g, b, 0, st, in, si, ldi, E, se, scale, ssc, out, so, ldo, kin, kout, len, batch);
  else if (kin <= 32) hipLaunchKernelGGL((rotate_kernel<32>), g, b, 0, st, in, si, ldi, E, se, scale, ssc, out, so, ldo, kin, kout, len, batch);
  else hipLaunchKernelGGL((rotate_kernel<64>), g, b, 0, st, in, si, ldi, E, se, scale, ssc, out, so, ldo, kin, kout, len, batch);
}

template <typename TX, typename TO, bool ACC64 = false>
void lowrank(const LowRankArgs& a, hipStream_t st) {
  ProfScope ps(SD_STAGE_LOWRANK, st);
  const dim3 g((a.rows_pad / 128) * (a.cols_pad / 128) * a.batch), b(256);
  if constexpr (ACC64) {
    if (a.kmax <= 16) hipLaunchKernelGGL((lowrank_kernel<TX, TO, 16, 1, true>), g, b, 0, st, a);
    else if (a.kmax <= 32) hipLaunchKernelGGL((lowrank_kernel<TX, TO, 32, 1, true>), g, b, 0, st, a);
    else hipLaunchKernelGGL((lowrank_kernel<TX, TO, 64, 1, true>), g, b, 0, st, a);
    return;
  }
  if (a.kmax <= 16) {
    if constexpr (sizeof(TX) == 2) hipLaunchKernelGGL((lowrank_kernel<TX, TO, 16, 4>), g, b, 0, st, a);
    else hipLaunchKernelGGL((lowrank_kernel<TX, TO, 16>), g, b, 0, st, a);
  }
  else if (a.kmax <= 32) hipLaunchKernelGGL((lowrank_kernel<TX, TO, 32>), g, b, 0, st, a);
  else hipLaunchKernelGGL((lowrank_kernel<TX, TO, 64>), g, b, 0, st, a);
}

}  // namespace sd
