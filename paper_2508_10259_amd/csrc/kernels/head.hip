// Action head, last stage: the bin logits (the last n_bins rows of the output
// head, computed by the projection GEMV after the final RMSNorm) reduced by a
// wavefront-shuffle argmax with the lowest bin winning ties; outputs, and the
// fed-back bin's embedding as the next decode pass's input.  One workgroup
// per row.
#include "common.h"
#include "kernels.h"

namespace ams {

// Argmax + outputs + feedback over precomputed bin logits (one workgroup per row).
template <typename T>
__global__ __launch_bounds__(256) void k_argmax_feed(const float* __restrict__ logits, int ldl, const T* __restrict__ bin_embed,
                                                     int d, int n_bins, int A, int j, int32_t* __restrict__ out_tok,
                                                     float* __restrict__ out_logits, const int32_t* __restrict__ forced,
                                                     float* __restrict__ h, int feed, T* __restrict__ h16,
                                                     T* __restrict__ h16lo) {
  __shared__ float red[16];
  __shared__ int redi[16];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const float* lg = logits + (size_t)b * ldl;
  const size_t oj = (size_t)b * A + j;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int bin = tid; bin < n_bins; bin += blockDim.x) {
    const float v = lg[bin];
    if (out_logits) out_logits[oj * n_bins + bin] = v;
    if (v > bv) { bv = v; bi = bin; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  if (lane == 0) { red[wave] = bv; redi[wave] = bi; }
  __syncthreads();
  bv = red[0];
  bi = redi[0];
  for (int w = 1; w < nw; ++w)
    if (red[w] > bv || (red[w] == bv && redi[w] < bi)) { bv = red[w]; bi = redi[w]; }
  if (bi < 0 || bi >= n_bins) bi = 0;  // every logit NaN
  if (tid == 0) out_tok[oj] = bi;
  if (feed) {
    int t = forced ? forced[oj] : bi;
    t = t < 0 ? 0 : (t >= n_bins ? n_bins - 1 : t);
    const T* e = bin_embed + (size_t)t * d;
    float* dst = h + (size_t)b * d;
    for (int i = tid; i < d; i += blockDim.x) dst[i] = ld<T>(e, i);
    if (h16) {  // the embedding row is already in the compute type: its pair is (e, 0)
      T* dst16 = h16 + (size_t)b * d;
      for (int i = tid; i < d; i += blockDim.x) dst16[i] = e[i];
      if (h16lo) {
        T* dstlo = h16lo + (size_t)b * d;
        for (int i = tid; i < d; i += blockDim.x) dstlo[i] = T(0);
      }
    }
  }
}

hipError_t argmax_feed(int ct, const float* logits, int ld_logits, const void* bin_embed, int B, int d, int n_bins,
                       int A, int j, int32_t* out_tok, float* out_logits, const int32_t* forced, float* h, int feed,
                       hipStream_t s, void* h16, void* h16lo) {
  if (ct == DT_F32) {
    if (h16 || h16lo) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_argmax_feed<float>, dim3(B), dim3(256), 0, s, logits, ld_logits, (const float*)bin_embed, d,
                       n_bins, A, j, out_tok, out_logits, forced, h, feed, (float*)nullptr, (float*)nullptr);
  } else {
    if (h16lo && !h16) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_argmax_feed<f16>, dim3(B), dim3(256), 0, s, logits, ld_logits, (const f16*)bin_embed, d,
                       n_bins, A, j, out_tok, out_logits, forced, h, feed, (f16*)h16, (f16*)h16lo);
  }
  return hipGetLastError();
}

}  // namespace ams
