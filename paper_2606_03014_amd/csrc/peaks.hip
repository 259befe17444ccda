// Microbenchmarks of the two peaks the engine's kernels are measured
// against on this GPU: streaming HBM read bandwidth, and bf16 matrix-core
// throughput of the 32x32x16 MFMA (the form the compute-bound kernels use).
// They report what the hardware sustains, beside the published peaks.
#include "kernels.h"

namespace moa {

typedef unsigned int pk_u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 pk_bf16x8 __attribute__((ext_vector_type(8)));
typedef float pk_f32x16 __attribute__((ext_vector_type(16)));

// Every byte of p[0, n) read once with 16-byte loads, eight in flight per
// thread; a data-dependent store keeps the loads alive.
__global__ __launch_bounds__(256) void k_peak_read(const pk_u32x4* __restrict__ p, size_t n, unsigned* sink) {
  constexpr int U = 8;
  pk_u32x4 acc = {0u, 0u, 0u, 0u};
  const size_t stride = (size_t)gridDim.x * 256 * U;
  for (size_t i = (size_t)blockIdx.x * 256 * U + threadIdx.x; i < n; i += stride) {
    pk_u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = (i + (size_t)u * 256 < n) ? p[i + (size_t)u * 256] : pk_u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u];
  }
  const unsigned x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (x == 0x9E3779B9u) sink[blockIdx.x] = x;
}

// Four independent accumulation chains of v_mfma_f32_32x32x16_bf16 per wave.
__global__ __launch_bounds__(256) void k_peak_mfma(float* sink, int iters, float seed) {
  const float a0 = seed * (float)(threadIdx.x & 63);
  pk_bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(a0 + (float)i);
    b[i] = (__bf16)(a0 - (float)i);
  }
  pk_f32x16 acc[4] = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  sink[blockIdx.x * 256 + threadIdx.x] = acc[0][0] + acc[1][5] + acc[2][10] + acc[3][15];
}

hipError_t launch_peak_read(hipStream_t st, const void* p, size_t bytes, unsigned* sink, int grid) {
  if (bytes < 16 || grid < 1) return hipErrorInvalidValue;
  k_peak_read<<<grid, 256, 0, st>>>((const pk_u32x4*)p, bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_peak_mfma(hipStream_t st, float* sink, int grid, int iters) {
  if (grid < 1 || iters < 1) return hipErrorInvalidValue;
  k_peak_mfma<<<grid, 256, 0, st>>>(sink, iters, 1e-3f);
  return hipGetLastError();
}

}  // namespace moa
