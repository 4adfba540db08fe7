// Test-only C ABI over single kernels (libams_probe.so), used by the GPU
// kernel tests to check one launcher at a time against plain definitions.
// Not part of the product library; the decoder's ABI is include/ams.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

extern "C" {

int ams_probe_gemm(int dtype, int epi, const void* u, const void* ulo, const void* W, int M, int N, int K, void* out,
                   int ldo, void* o16, void* olo, void* stream) {
  return (int)ams::gemm(dtype, epi, u, W, M, N, K, out, ldo, (hipStream_t)stream, ulo, o16, olo);
}

int ams_probe_gemm_big(int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo, int bn,
                       void* stream) {
  return (int)ams::gemm_big(epi, u, W, M, N, K, out, ldo, (hipStream_t)stream, bn);
}

int ams_probe_gemm_big_part(const void* u, const void* W, int M, int N, int K, int splits, float* part,
                            void* stream) {
  return (int)ams::gemm_big_part(u, W, M, N, K, splits, part, (hipStream_t)stream);
}

int ams_probe_gemm_part(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                        void* stream) {
  return (int)ams::gemm_part(u, ulo, W, M, N, K, splits, part, (hipStream_t)stream);
}

int ams_probe_part_resid(const float* part, int splits, int M, int N, float* h, void* o16, void* olo, void* stream) {
  return (int)ams::part_resid(part, splits, M, N, h, o16, olo, (hipStream_t)stream);
}

int ams_probe_frag_pack(const void* W, int N, int K, void* Wf, void* stream) {
  return (int)ams::frag_pack(W, N, K, Wf, (hipStream_t)stream);
}
int ams_probe_gemm_wide(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                        void* stream) {
  return (int)ams::gemm_wide(u, ulo, W, M, N, K, splits, part, (hipStream_t)stream);
}

int ams_probe_gemm_wide_reduce(int epi, const void* u, const void* ulo, const void* W, int M, int N, int K,
                               int splits, float* part, unsigned* counters, void* out, void* olo, int ldo, float* h,
                               void* o16, void* olo2, float* ss_out, const float* ss_in, float eps, void* stream) {
  return (int)ams::gemm_wide_reduce(epi, u, ulo, W, M, N, K, splits, part, counters, out, olo, ldo, h, o16, olo2,
                                    ss_out, ss_in, eps, (hipStream_t)stream);
}

int ams_probe_part_store(const float* part, int splits, int M, int N, float* out, void* stream) {
  return (int)ams::part_store(part, splits, M, N, out, (hipStream_t)stream);
}
int ams_probe_part_resid_ss(const float* part, int splits, int M, int N, float* h, void* o16, void* olo, float* ss,
                            void* stream) {
  return (int)ams::part_resid(part, splits, M, N, h, o16, olo, (hipStream_t)stream, ss);
}
int ams_probe_part_store_norm(const float* part, int splits, int M, int N, float* out, const float* ss, int d,
                              float eps, void* stream) {
  return (int)ams::part_store(part, splits, M, N, out, (hipStream_t)stream, ss, d, eps);
}
int ams_probe_part_swiglu_norm(const float* part, int splits, int M, int N, void* out, void* olo, const float* ss,
                               int d, float eps, void* stream) {
  return (int)ams::part_swiglu(part, splits, M, N, out, olo, (hipStream_t)stream, ss, d, eps);
}

int ams_probe_part_swiglu(const float* part, int splits, int M, int N, void* out, void* olo, void* stream) {
  return (int)ams::part_swiglu(part, splits, M, N, out, olo, (hipStream_t)stream);
}

int ams_probe_resid_norm(const float* part, int splits, int M, int d, float* h, float eps, void* u, void* stream) {
  return (int)ams::resid_norm(part, splits, M, d, h, eps, u, (hipStream_t)stream);
}

int ams_probe_rmsnorm(int dtype, const float* h, int M, int d, float eps, void* u, void* ulo, void* stream) {
  return (int)ams::rmsnorm(dtype, h, M, d, eps, u, (hipStream_t)stream, ulo);
}

int ams_probe_argmax_feed(int ct, const float* logits, int ld, const void* bin_embed, int B, int d, int n_bins,
                          int A, int j, int32_t* out_tok, float* out_logits, const int32_t* forced, float* h, int feed,
                          void* h16, void* h16lo, void* stream) {
  return (int)ams::argmax_feed(ct, logits, ld, bin_embed, B, d, n_bins, A, j, out_tok, out_logits, forced, h, feed,
                               (hipStream_t)stream, h16, h16lo);
}

int ams_probe_gemv_rmsnorm(int ct, int epi, const void* hhi, const void* hlo, float eps, const void* W, int M, int N,
                           int K, void* out, int ldo, void* o16, void* olo, void* stream) {
  return (int)ams::gemv_rmsnorm(ct, epi, hhi, eps, W, M, N, K, out, ldo, (hipStream_t)stream, hlo, o16, olo);
}

// decode attention of one pass (jpos) for B rows, merged when splits > 1; K/V in
// page pools [page][H][64][dh] with row b's page table at pt + b * (cap / 64)
// (order: NULL or the rows' dispatch order, see len_order)
int ams_probe_attn_decode(int ct, const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh, int cap,
                          const int32_t* pt, int splits, const void* rope, void* kslab, void* vslab, float* part,
                          void* o, void* olo, const int32_t* order, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = ams::attn_decode(ct, qkv, lens, jpos, B, H, dh, cap, ams::KvPages{pt, cap / 64}, splits,
                                  (const float2*)rope, kslab, vslab, part, o, s, olo, ams::QkvParts{}, order);
  if (e == hipSuccess && splits > 1) e = ams::attn_merge(ct, part, B, H, dh, splits, o, s, olo);
  return (int)e;
}

int ams_probe_len_order(const int32_t* lens, int B, int32_t* order, void* stream) {
  return (int)ams::len_order(lens, B, order, (hipStream_t)stream);
}

// Causal attention of packed segments (row[s], pos[s], off[s..s+1]) over their rows' K/V pages.
int ams_probe_attn_decode_parts(int ct, const float* qpart, int qsplits, const float* ss, int nss, float eps,
                                const int32_t* lens, int jpos, int B, int H, int dh, int cap, const int32_t* pt,
                                int splits, const void* rope, void* kslab, void* vslab, float* part, void* o, void* olo,
                                void* stream) {
  hipStream_t s = (hipStream_t)stream;
  ams::QkvParts qp;
  qp.part = qpart;
  qp.splits = qsplits;
  qp.ss = ss;
  qp.nss = nss;
  qp.eps = eps;
  hipError_t e = ams::attn_decode(ct, qpart, lens, jpos, B, H, dh, cap, ams::KvPages{pt, cap / 64}, splits,
                                  (const float2*)rope, kslab, vslab, part, o, s, olo, qp);
  if (e == hipSuccess && splits > 1) e = ams::attn_merge(ct, part, B, H, dh, splits, o, s, olo);
  return (int)e;
}

// K/V append of a pass's tokens, and the QKV GEMM with the append in its epilogue
// (token tables into tok_base / tok_pos first)
int ams_probe_kv_append(int ct, const float* qkv, const int32_t* row, const int32_t* pos, const int32_t* off,
                        int n_seg, int n_tok, int max_len, int max_end, int H, int dh, int cap, const int32_t* pt,
                        const void* rope, void* kslab, void* vslab, void* stream) {
  ams::Segs sg{row, pos, off, n_seg, n_tok, max_len, max_end};
  return (int)ams::kv_append(ct, qkv, sg, H, dh, ams::KvPages{pt, cap / 64}, (const float2*)rope, kslab, vslab,
                             (hipStream_t)stream);
}
int ams_probe_kv_append_tab(const float* qkv, const int32_t* row, const int32_t* pos, const int32_t* off, int n_seg,
                            int n_tok, int H, int dh, int cap, const int32_t* pt, const void* rope, void* kslab,
                            void* vslab, int64_t* tok_base, int32_t* tok_pos, void* stream) {
  ams::Segs sg{row, pos, off, n_seg, n_tok, 0, 0};
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = ams::tok_tables(sg, ams::KvPages{pt, cap / 64}, H, dh, tok_base, tok_pos, s);
  if (e == hipSuccess) e = ams::kv_append_tab(qkv, n_tok, tok_base, tok_pos, H, dh, (const float2*)rope, kslab, vslab, s);
  return (int)e;
}
int ams_probe_qkv_kv(const void* u, const void* W, int K, float* qkv, const int32_t* row, const int32_t* pos,
                     const int32_t* off, int n_seg, int n_tok, int H, int dh, int cap, const int32_t* pt,
                     const void* rope, void* kslab, void* vslab, int64_t* tok_base, int32_t* tok_pos, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  ams::Segs sg{row, pos, off, n_seg, n_tok, 0, 0};
  ams::KvPages kp{pt, cap / 64};
  hipError_t e = ams::tok_tables(sg, kp, H, dh, tok_base, tok_pos, s);
  if (e != hipSuccess) return (int)e;
  ams::KvEpi kv{tok_base, tok_pos, kslab, vslab, (const float2*)rope, H * dh, dh};
  return (int)ams::gemm_qkv_kv(u, W, n_tok, K, qkv, kv, s);
}
int ams_probe_qkv_fusable(int M, int N, int dh, int d) { return ams::gemm_qkv_fusable(M, N, dh, d) ? 1 : 0; }

int ams_probe_attn_prefill(int ct, const float* qkv, const int32_t* row, const int32_t* pos, const int32_t* off,
                           int n_seg, int n_tok, int max_len, int max_end, int H, int dh, int cap, const int32_t* pt,
                           const void* rope, const void* kslab, const void* vslab, void* o, void* stream) {
  ams::Segs sg{row, pos, off, n_seg, n_tok, max_len, max_end};
  return (int)ams::attn_prefill(ct, qkv, sg, H, dh, ams::KvPages{pt, cap / 64}, (const float2*)rope, kslab, vslab, o,
                                (hipStream_t)stream);
}

int ams_probe_stream_copy(const void* src, void* dst, size_t bytes, int grid, void* stream) {
  return (int)ams::stream_copy(src, dst, bytes, grid, (hipStream_t)stream);
}

int ams_probe_stream_read(const void* src, size_t bytes, float* out, int grid, void* stream) {
  return (int)ams::stream_read(src, bytes, out, grid, (hipStream_t)stream);
}

int ams_probe_mfma_loop(int shape, float x, int iters, float* out, int grid, void* stream) {
  return (int)ams::mfma_loop(shape, x, iters, out, grid, (hipStream_t)stream);
}

double ams_probe_mfma_loop_flops(int iters, int grid) { return ams::mfma_loop_flops(iters, grid); }

}  // extern "C"
