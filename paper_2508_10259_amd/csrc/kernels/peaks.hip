// Measured peaks of the two roofs the hot path is judged against: HBM stream
// bandwidth (a copy and a read of buffers far larger than the 256 MB memory-side
// cache) and the dense fp16 MFMA rate (register-only MFMA chains on every SIMD).
// The decoder does not use them; they give the measured denominators beside the
// published 8 TB/s and 2.5 PFLOP/s.
#include "common.h"
#include "kernels.h"

namespace ams {

namespace {

__global__ __launch_bounds__(256) void k_stream_copy(const float4* __restrict__ src, float4* __restrict__ dst,
                                                     size_t n4) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_stream_read(const float4* __restrict__ src, size_t n4,
                                                     float* __restrict__ out) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  float a = 0.f;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 v = src[i];
    a += (v.x + v.y) + (v.z + v.w);
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = a;
}

// Register-only MFMA chains on every SIMD (operands all x): SHAPE 0 runs 8
// independent chains of v_mfma_f32_16x16x32_f16, SHAPE 1 4 chains of
// v_mfma_f32_32x32x16_f16 -- the same 131072 FLOP per wave and round, and each
// lane ends with the sum of its accumulators, 1024 x^2 per round.
constexpr int MFMA_CHAINS = 8;
typedef float f32x16 __attribute__((ext_vector_type(16)));
template <int SHAPE>
__global__ __launch_bounds__(256) void k_mfma_loop(float x, int iters, float* __restrict__ out) {
  const f16 hx = (f16)x;
  const half8 a = {hx, hx, hx, hx, hx, hx, hx, hx};
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    // the chains in inline assembly, each accumulator updated in place (written
    // as builtins the compiler moved accumulators between registers every round)
    f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
    for (int it = 0; it < iters; ++it) {
      asm volatile(
          "v_mfma_f32_16x16x32_f16 %0, %8, %8, %0\n\t"
          "v_mfma_f32_16x16x32_f16 %1, %8, %8, %1\n\t"
          "v_mfma_f32_16x16x32_f16 %2, %8, %8, %2\n\t"
          "v_mfma_f32_16x16x32_f16 %3, %8, %8, %3\n\t"
          "v_mfma_f32_16x16x32_f16 %4, %8, %8, %4\n\t"
          "v_mfma_f32_16x16x32_f16 %5, %8, %8, %5\n\t"
          "v_mfma_f32_16x16x32_f16 %6, %8, %8, %6\n\t"
          "v_mfma_f32_16x16x32_f16 %7, %8, %8, %7"
          : "+a"(c0), "+a"(c1), "+a"(c2), "+a"(c3), "+a"(c4), "+a"(c5), "+a"(c6), "+a"(c7)
          : "v"(a));
    }
    asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");  // results of the last MFMAs ready before they are read
    const f32x4 t = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));
    s = (t[0] + t[1]) + (t[2] + t[3]);
  } else {
    f32x16 acc[MFMA_CHAINS / 2];
#pragma unroll
    for (int j = 0; j < MFMA_CHAINS / 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < MFMA_CHAINS / 2; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, a, acc[j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < MFMA_CHAINS / 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; e += 4) s += (acc[j][e] + acc[j][e + 1]) + (acc[j][e + 2] + acc[j][e + 3]);
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

hipError_t stream_copy(const void* src, void* dst, size_t bytes, int grid, hipStream_t s) {
  if (bytes % 16 != 0 || grid < 1 || ((uintptr_t)src | (uintptr_t)dst) % 16 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_stream_copy, dim3(grid), dim3(256), 0, s, (const float4*)src, (float4*)dst, bytes / 16);
  return hipGetLastError();
}

hipError_t stream_read(const void* src, size_t bytes, float* out, int grid, hipStream_t s) {
  if (bytes % 16 != 0 || grid < 1 || (uintptr_t)src % 16 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_stream_read, dim3(grid), dim3(256), 0, s, (const float4*)src, bytes / 16, out);
  return hipGetLastError();
}

hipError_t mfma_loop(int shape, float x, int iters, float* out, int grid, hipStream_t s) {
  if (iters < 1 || grid < 1 || (shape != 0 && shape != 1)) return hipErrorInvalidValue;
  if (shape == 0) hipLaunchKernelGGL(k_mfma_loop<0>, dim3(grid), dim3(256), 0, s, x, iters, out);
  else hipLaunchKernelGGL(k_mfma_loop<1>, dim3(grid), dim3(256), 0, s, x, iters, out);
  return hipGetLastError();
}

double mfma_loop_flops(int iters, int grid) {
  return (double)grid * (256 / 64) * iters * MFMA_CHAINS * (16.0 * 16.0 * 32.0 * 2.0);
}

}  // namespace ams
