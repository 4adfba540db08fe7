// Flow-matching action head over a cached context (paper section 3.2.1: the
// diffusion model's latent vectors are part of the action context; section
// 3.4.2, Action Regeneration: sampling restarts from a stored latent).
//
// One Euler step of the latent x [token][a] of every row's action chunk:
//   k_flow_embed:  h[t] = W_in x[t] + tau w_t      (the chunk's tokens enter the decoder)
//   (every decoder layer over the tokens, at the positions after each row's context)
//   k_flow_update: x[t] += dt W_out (h[t] / rms(h[t]))
// Both are small per-token kernels around the decoder's token pass; the pass
// itself (GEMMs on MFMA, attention over the cached K/V pages) is the same code
// that builds and extends contexts.
#include "common.h"
#include "kernels.h"

namespace ams {

namespace {

// One workgroup per token: x of the token in LDS, one output dimension per thread.
template <typename T>
__global__ __launch_bounds__(256) void k_flow_embed(const float* __restrict__ x, const T* __restrict__ w_in,
                                                    const T* __restrict__ w_t, float tau, int a, int d,
                                                    float* __restrict__ h) {
  __shared__ float xs[FLOW_MAX_ACTION_DIM];
  const int t = blockIdx.x;
  for (int k = threadIdx.x; k < a; k += blockDim.x) xs[k] = x[(size_t)t * a + k];
  __syncthreads();
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    float e = tau * ld<T>(w_t, j);
    for (int k = 0; k < a; ++k) e = fmaf(ld<T>(w_in, (size_t)j * a + k), xs[k], e);
    h[(size_t)t * d + j] = e;
  }
}

// One workgroup per token: the RMS of h, then one output per wave at a time (a
// dot product over d with lane-strided loads and a wavefront sum).
template <typename T>
__global__ __launch_bounds__(256) void k_flow_update(const float* __restrict__ h, const T* __restrict__ w_out,
                                                     float eps, float dt, int a, int d, float* __restrict__ x) {
  __shared__ float red[16];
  const int t = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const float* ht = h + (size_t)t * d;
  float ss = 0.f;
  for (int j = threadIdx.x; j < d; j += blockDim.x) ss = fmaf(ht[j], ht[j], ss);
  const float r = rsqrtf(block_sum(ss, red) / (float)d + eps);
  for (int i = wave; i < a; i += nw) {
    float v = 0.f;
    for (int j = lane; j < d; j += 64) v = fmaf(ld<T>(w_out, (size_t)i * d + j), ht[j], v);
    v = wave_sum(v);
    if (lane == 0) x[(size_t)t * a + i] += dt * (v * r);
  }
}

}  // namespace

hipError_t flow_embed(int st, const float* x, const void* w_in, const void* w_t, float tau, int n_tok, int a, int d,
                      float* h, hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  if (a < 1 || a > FLOW_MAX_ACTION_DIM) return hipErrorInvalidValue;
  if (st == DT_F32)
    hipLaunchKernelGGL(k_flow_embed<float>, dim3(n_tok), dim3(256), 0, s, x, (const float*)w_in, (const float*)w_t,
                       tau, a, d, h);
  else
    hipLaunchKernelGGL(k_flow_embed<bf16>, dim3(n_tok), dim3(256), 0, s, x, (const bf16*)w_in, (const bf16*)w_t,
                       tau, a, d, h);
  return hipGetLastError();
}

hipError_t flow_update(int st, const float* h, const void* w_out, float eps, float dt, int n_tok, int a, int d,
                       float* x, hipStream_t s) {
  if (n_tok <= 0) return hipSuccess;
  if (st == DT_F32)
    hipLaunchKernelGGL(k_flow_update<float>, dim3(n_tok), dim3(256), 0, s, h, (const float*)w_out, eps, dt, a, d, x);
  else
    hipLaunchKernelGGL(k_flow_update<bf16>, dim3(n_tok), dim3(256), 0, s, h, (const bf16*)w_out, eps, dt, a, d, x);
  return hipGetLastError();
}

}  // namespace ams
