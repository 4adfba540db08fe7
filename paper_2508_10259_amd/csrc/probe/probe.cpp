// Test-only C ABI over single kernels (libams_probe.so), used by the GPU
// kernel tests to check one launcher at a time against plain definitions.
// Not part of the product library; the decoder's ABI is include/ams.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

extern "C" {

int ams_probe_gemm(int dtype, int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo,
                   void* out16, void* stream) {
  return (int)ams::gemm(dtype, epi, u, W, M, N, K, out, ldo, (hipStream_t)stream, out16);
}

int ams_probe_rmsnorm(int dtype, const float* h, int M, int d, float eps, void* u, void* stream) {
  return (int)ams::rmsnorm(dtype, h, M, d, eps, u, (hipStream_t)stream);
}

int ams_probe_argmax_feed(int ct, const float* logits, int ld, const void* bin_embed, int B, int d, int n_bins,
                          int A, int j, int32_t* out_tok, float* out_logits, const int32_t* forced, float* h, int feed,
                          void* h16, void* stream) {
  return (int)ams::argmax_feed(ct, logits, ld, bin_embed, B, d, n_bins, A, j, out_tok, out_logits, forced, h, feed,
                               (hipStream_t)stream, h16);
}

int ams_probe_gemv_rmsnorm(int ct, int epi, const void* h16, float eps, const void* W, int M, int N, int K, void* out,
                           int ldo, void* out16, void* stream) {
  return (int)ams::gemv_rmsnorm(ct, epi, h16, eps, W, M, N, K, out, ldo, (hipStream_t)stream, out16);
}

}  // extern "C"
