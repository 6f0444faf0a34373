// Peak-rate microbenchmarks behind the roofline constants the benchmark
// prices against, re-measured on the device: dense bf16 MFMA throughput
// (v_mfma_f32_32x32x16_bf16 on register operands, eight independent
// accumulators per wave) and HBM streaming bandwidth (a float4 copy and a
// float4 read-and-reduce over buffers far larger than the caches). C entry
// points; the caller times them.
#include <hip/hip_runtime.h>
#include <stddef.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

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

__global__ __launch_bounds__(256) void sdp_copy_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                                       size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ __launch_bounds__(256) void sdp_read_kernel(const float4* __restrict__ src, size_t n, float* sink) {
  float s = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const float4 v = src[i];
    s += v.x + v.y + v.z + v.w;
  }
  if (s == -1.0f) sink[blockIdx.x] = s;
}

extern "C" {
// flops of one sdp_mfma_bf16 launch: blocks * 4 waves * 8 * iters * 32768
int sdp_mfma_bf16(int blocks, int iters, float* sink, hipStream_t stream) {
  if (blocks < 1 || iters < 1 || !sink) return -1;
  hipLaunchKernelGGL(sdp_mfma_bf16_kernel, dim3(blocks), dim3(256), 0, stream, iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
// n float4 elements each way (src and dst do not overlap)
int sdp_copy(const void* src, void* dst, size_t n, int blocks, hipStream_t stream) {
  if (!src || !dst || n == 0 || blocks < 1) return -1;
  hipLaunchKernelGGL(sdp_copy_kernel, dim3(blocks), dim3(256), 0, stream, (const float4*)src, (float4*)dst, n);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
int sdp_read(const void* src, size_t n, int blocks, float* sink, hipStream_t stream) {
  if (!src || n == 0 || blocks < 1 || !sink) return -1;
  hipLaunchKernelGGL(sdp_read_kernel, dim3(blocks), dim3(256), 0, stream, (const float4*)src, n, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
}
