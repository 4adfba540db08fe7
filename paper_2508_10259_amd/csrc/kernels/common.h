// Device-side helpers shared by the CDNA4 (gfx950) kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ams {

// bf16 values (the caller's storage type) are carried as raw 16-bit patterns.
typedef uint16_t bf16;
// fp16: the compute type of bf16-stored models (MFMA inputs, activations, K/V).
typedef _Float16 f16;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float F16_MAX = 65504.0f;

__device__ __forceinline__ float bf2f(bf16 b) { return __uint_as_float(((uint32_t)b) << 16); }

// Round to nearest, ties to even (finite inputs).
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
}

// 16 bytes of a stream read once per launch (weights of a decode GEMV, the K/V
// cache under a decode or extension attention), as a non-temporal load: the
// stream does not push out what other workgroups re-read from L2 and the
// Infinity Cache (the activations, the split-K partial sums, the page tables).
__device__ __forceinline__ uint4 ld_stream(const void* p) {
  typedef unsigned u32x4s __attribute__((ext_vector_type(4)));
  const u32x4s x = __builtin_nontemporal_load((const u32x4s*)p);
  return uint4{x[0], x[1], x[2], x[3]};
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16> {
  static __device__ __forceinline__ float load(const bf16* p, size_t i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void store(bf16* p, size_t i, float v) { p[i] = f2bf(v); }
};
// fp16 stores saturate at the largest finite value instead of overflowing to inf.
template <> struct Elem<f16> {
  static __device__ __forceinline__ float load(const f16* p, size_t i) { return (float)p[i]; }
  static __device__ __forceinline__ void store(f16* p, size_t i, float v) {
    p[i] = (f16)fminf(fmaxf(v, -F16_MAX), F16_MAX);
  }
};

template <typename T> __device__ __forceinline__ float ld(const T* p, size_t i) { return Elem<T>::load(p, i); }
template <typename T> __device__ __forceinline__ void st(T* p, size_t i, float v) { Elem<T>::store(p, i, v); }

// fp16 pair of v: hi[i] = fp16(v) (saturating), lo[i] = fp16(v - hi[i]) when lo
// is non-NULL; hi + lo carries about 22 significant bits of v.
__device__ __forceinline__ f16 sat16(float v) { return (f16)fminf(fmaxf(v, -F16_MAX), F16_MAX); }
__device__ __forceinline__ void split16(float v, f16* hi, f16* lo, size_t i) {
  const f16 h = sat16(v);
  hi[i] = h;
  if (lo) lo[i] = sat16(v - (float)h);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum over a whole workgroup of `nthreads` (multiple of 64, <= 1024); `red`
// is LDS scratch of >= 16 floats.  Every thread gets the total.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// Load of an int that stays constant while the kernel runs (a page-table
// entry), at a wave-uniform address: read through the constant address space
// so that it becomes a scalar load served by the scalar cache.
__device__ __forceinline__ int ld_const_uniform(const int32_t* p, size_t i) {
  typedef const int32_t __attribute__((address_space(4))) cint;
  return ((cint*)p)[i];
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + __expf(-z)); }

}  // namespace ams
