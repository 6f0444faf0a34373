// Peak-rate microbenchmarks behind the roofline constants the benchmark
// prices against, re-measured on the device: dense bf16 MFMA throughput
// (v_mfma_f32_32x32x16_bf16 on register operands, eight independent
// accumulators per wave) and HBM streaming bandwidth (a float4 copy and a
// float4 read-and-reduce over buffers far larger than the caches, each in a
// grid-stride and a chunk-per-work-group form). C entry points; the caller
// times them.
#include <hip/hip_runtime.h>
#include <stddef.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Each wave issues 8 * iters MFMAs of 32 x 32 x 16 (32768 flops each). The
// results feed a comparison that is never true in practice, so the products
// are not removed, and nothing is stored unless it is.
__global__ __launch_bounds__(256) void sdp_mfma_bf16_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.001f * (float)((lane * 3 + i) & 7));
  }
  f32x16_t c[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) c[j] = f32x16_t{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[j][e];
  if (s == -1.0f) sink[blockIdx.x] = s;
}

// Streaming kernels: every thread moves U consecutive-stride float4 per
// iteration with all loads issued before the stores (more bytes in flight);
// the copy's stores are non-temporal. n is a multiple of the grid's stride
// times U (the caller sizes the buffers so).
constexpr int STREAM_U = 4;
__global__ __launch_bounds__(256) void sdp_copy_kernel(const f32x4_t* __restrict__ src, f32x4_t* __restrict__ dst,
                                                       size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride * STREAM_U) {
    f32x4_t v[STREAM_U];
#pragma unroll
    for (int u = 0; u < STREAM_U; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < STREAM_U; ++u) __builtin_nontemporal_store(v[u], &dst[i + u * stride]);
  }
}

__global__ __launch_bounds__(256) void sdp_read_kernel(const float4* __restrict__ src, size_t n, float* sink) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  float s = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride * STREAM_U) {
    float4 v[STREAM_U];
#pragma unroll
    for (int u = 0; u < STREAM_U; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < STREAM_U; ++u) s += v[u].x + v[u].y + v[u].z + v[u].w;
  }
  if (s == -1.0f) sink[blockIdx.x] = s;
}

// The same streams with one contiguous chunk of 256 U float4 per work-group
// (every load of the chunk in flight before its first use; a grid of n /
// (256 U) work-groups, n a multiple of 256 U): whole DRAM pages per work-group
// instead of the grid-stride pattern above, and, for the read, optionally
// non-temporal loads.
template <bool NT>
__global__ __launch_bounds__(256) void sdp_read_chunk_kernel(const f32x4_t* __restrict__ src, float* sink) {
  const f32x4_t* p = src + (size_t)blockIdx.x * 256 * STREAM_U + threadIdx.x;
  f32x4_t v[STREAM_U];
#pragma unroll
  for (int u = 0; u < STREAM_U; ++u) v[u] = NT ? __builtin_nontemporal_load(p + u * 256) : p[u * 256];
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < STREAM_U; ++u) s += v[u][0] + v[u][1] + v[u][2] + v[u][3];
  if (s == -1.0f) sink[blockIdx.x] = s;
}
__global__ __launch_bounds__(256) void sdp_copy_chunk_kernel(const f32x4_t* __restrict__ src,
                                                             f32x4_t* __restrict__ dst) {
  const size_t o = (size_t)blockIdx.x * 256 * STREAM_U + threadIdx.x;
  f32x4_t v[STREAM_U];
#pragma unroll
  for (int u = 0; u < STREAM_U; ++u) v[u] = src[o + u * 256];
#pragma unroll
  for (int u = 0; u < STREAM_U; ++u) __builtin_nontemporal_store(v[u], &dst[o + u * 256]);
}

extern "C" {
// flops of one sdp_mfma_bf16 launch: blocks * 4 waves * 8 * iters * 32768
int sdp_mfma_bf16(int blocks, int iters, float* sink, hipStream_t stream) {
  if (blocks < 1 || iters < 1 || !sink) return -1;
  hipLaunchKernelGGL(sdp_mfma_bf16_kernel, dim3(blocks), dim3(256), 0, stream, iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
// n float4 elements each way (src and dst do not overlap); n must be a
// multiple of blocks * 256 * 4
int sdp_copy(const void* src, void* dst, size_t n, int blocks, hipStream_t stream) {
  if (!src || !dst || n == 0 || blocks < 1 || n % ((size_t)blocks * 256 * STREAM_U)) return -1;
  hipLaunchKernelGGL(sdp_copy_kernel, dim3(blocks), dim3(256), 0, stream, (const f32x4_t*)src, (f32x4_t*)dst, n);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
int sdp_read(const void* src, size_t n, int blocks, float* sink, hipStream_t stream) {
  if (!src || n == 0 || blocks < 1 || !sink || n % ((size_t)blocks * 256 * STREAM_U)) return -1;
  hipLaunchKernelGGL(sdp_read_kernel, dim3(blocks), dim3(256), 0, stream, (const float4*)src, n, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
// Chunked forms: n float4 elements, a multiple of 256 * 4; the grid is n / 1024
// work-groups (at most 2^31 - 1), so sink must hold n / 1024 floats.
int sdp_copy_chunk(const void* src, void* dst, size_t n, hipStream_t stream) {
  const size_t chunk = (size_t)256 * STREAM_U;
  if (!src || !dst || n == 0 || n % chunk || n / chunk > 0x7fffffffull) return -1;
  hipLaunchKernelGGL(sdp_copy_chunk_kernel, dim3((unsigned)(n / chunk)), dim3(256), 0, stream, (const f32x4_t*)src,
                     (f32x4_t*)dst);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
int sdp_read_chunk(const void* src, size_t n, int nontemporal, float* sink, hipStream_t stream) {
  const size_t chunk = (size_t)256 * STREAM_U;
  if (!src || !sink || n == 0 || n % chunk || n / chunk > 0x7fffffffull) return -1;
  const dim3 g((unsigned)(n / chunk));
  if (nontemporal) hipLaunchKernelGGL(sdp_read_chunk_kernel<true>, g, dim3(256), 0, stream, (const f32x4_t*)src, sink);
  else hipLaunchKernelGGL(sdp_read_chunk_kernel<false>, g, dim3(256), 0, stream, (const f32x4_t*)src, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
}
