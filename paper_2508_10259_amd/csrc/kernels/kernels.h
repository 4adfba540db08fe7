// Host-side launchers of the gfx950 kernels.  Every launcher only enqueues
// on the given stream and returns the launch status; argument validation
// happens in the C ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fused_limits.h"

namespace ams {

// Storage types at the boundary: DT_F32, DT_BF16.  Compute types inside the
// kernels (GEMM inputs, activations, K/V slab, packed weights): DT_F32 for
// fp32 models, DT_F16 for bf16 models.
enum DType { DT_F32 = 0, DT_BF16 = 1, DT_F16 = 2 };
enum Epi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_PART = 3 /* internal: split-K partial sums */,
           EPI_QKV = 4 /* internal: QKV projection with RoPE + K/V append */ };

// Packed-token pass metadata (device arrays).  Segment s covers tokens
// off[s]..off[s+1]-1 of the pass, which belong to row `row[s]` at positions
// pos[s], pos[s]+1, ...
// K/V of a context, per layer: K and V each a pool of pages [page][head][64][head_dim]
// (model compute type).  Row b's position t sits in page pt[b * ppr + t / 64] at
// slot t % 64; pt is a device int32 array [rows][ppr].  Rows whose inputs agree
// up to a page's end may point at the same page.
constexpr int KV_PAGE = 64;
struct KvPages {
  const int32_t* pt;
  int ppr;  // pages per row (capacity / 64)
};

struct Segs {
  const int32_t* row;
  const int32_t* pos;
  const int32_t* off;  // n_seg + 1 entries
  int n_seg;
  int n_tok;
  int max_len;  // longest segment
  int max_end;  // largest pos[s] + len(s)
  // NULL, or the pass's segments longest attention first (pos + len decreasing):
  // the extension attention dispatches its workgroups in that order
  const int32_t* order = nullptr;
};

// Gate/up rows are packed interleaved in blocks of 16: packed row 32i+j is
// gate row 16i+j for j < 16 and up row 16i+j-16 otherwise, so a 32-row strip
// holds the gate and up rows of the same 16 SwiGLU outputs.
constexpr int GU_BLOCK = 16;

// y[m][n] = sum_k u[m][k] * W[n][k] followed by the epilogue:
//   EPI_STORE : out_f32[m*ldo + n] = y
//   EPI_RESID : out_f32[m*ldo + n] += y          (residual stream)
//   EPI_SWIGLU: out_T[m*ldo + c] = silu(gate_c) * up_c with W packed as above
// fp16-pair forms (fp16 compute, M <= 64 only; NULL otherwise):
//   ulo : the input is u + ulo (ulo = the rounding error of u, same shape)
//   o16 : EPI_RESID also writes the updated rows as fp16 (saturating), same ldo
//   olo : the rounding error of o16 (EPI_RESID) or of the fp16 out (EPI_SWIGLU)
hipError_t gemm(int ct, int epi, const void* u, const void* W, int M, int N, int K, void* out,
                int ldo, hipStream_t s, const void* ulo = nullptr, void* o16 = nullptr, void* olo = nullptr);

// Split-K decode GEMV (fp16, M <= 64): part[s][m][n] = sum over the s-th of
// `splits` equal K ranges (in 128-wide chunks) of u[m][k] W[n][k], with u the
// fp16 input or the pair u + ulo as in gemm().  part holds splits * M * N floats.
hipError_t gemm_part(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                     hipStream_t s);
// MFMA fragment order of an fp16 matrix W [N][K] (N a multiple of 16, K of
// 128): 16-row strip s, 128-column chunk c and 32-column step i of it form one
// 1 KB block, lane l of a wave holding row 16 s + l % 16, columns
// 128 c + 32 i + 8 (l / 16) .. +8:
//   Wf[(((s * K/128 + c) * 4 + i) * 64 + l) * 8 + e] = W[16 s + l % 16][128 c + 32 i + 8 (l / 16) + e]
// so a wave reads the A fragments of one MFMA step as 1 KB of contiguous memory.
hipError_t frag_pack(const void* W, int N, int K, void* Wf, hipStream_t s);

// Wide decode GEMM (fp16, 16 < M <= 64 typical, N a multiple of 128, W in
// fragment order): the same partial sums as gemm_part, with 128 weight rows
// per workgroup sharing LDS-staged activations.  The epilogue is one of the
// part_* reductions.
hipError_t gemm_wide(const void* u, const void* ulo, const void* W, int M, int N, int K, int splits, float* part,
                     hipStream_t s);
// The wide decode GEMM (W in fragment order) with its reduction fused: each
// split stores its partial sums (part, splits * M * N floats) and the last
// split of every 128-row weight tile to finish (per-tile counters, zero before
// the first call, left zero) adds them in split order and applies the
// epilogue, with the results of the part_* reductions:
//   EPI_STORE : out[m*ldo + n] = y / rms_m        (rms_m from ss_in, or 1 when NULL)
//   EPI_SWIGLU: out/olo[m*ldo + c] = silu(gate / rms_m) * (up / rms_m), fp16 pair
//   EPI_RESID : h[m][n] += y, the fp16 pair (o16, olo2) of the new rows when
//               o16 is non-NULL, and the sums of squares of the new rows per 128
//               columns in ss_out[m][n / 128] when non-NULL
// ss_in: sums of squares of the unnormalised input rows per 128 columns
// ([M][K / 128]), rms_m = sqrt(sum / K + eps).  counters: N / 128 entries.
hipError_t gemm_wide_reduce(int epi, const void* u, const void* ulo, const void* W, int M, int N, int K, int splits,
                            float* part, unsigned* counters, void* out, void* olo, int ldo, float* h, void* o16,
                            void* olo2, float* ss_out, const float* ss_in, float eps, hipStream_t s);
// out[m][n] = sum_s part[s][m][n] (fp32 out).  With ss (the sums of squares
// per 128 columns part_resid left for a residual of width d, both N and d
// multiples of 256)
// the GEMM read that residual unnormalised and row m is scaled by its
// 1/sqrt(sum/d + eps): RMSNorm(h) W^T = (h W^T) / rms(h), the gains being
// folded into W.
hipError_t part_store(const float* part, int splits, int M, int N, float* out, hipStream_t s,
                      const float* ss = nullptr, int d = 0, float eps = 0.f);
// out[m][c] = silu(gate) * up of the summed packed gate/up rows of column c
// (N = 2F packed rows), fp16 with its rounding error in olo (or NULL); ss,
// d, eps as for part_store (N / 2 a multiple of 256).
hipError_t part_swiglu(const float* part, int splits, int M, int N, void* out, void* olo, hipStream_t s,
                       const float* ss = nullptr, int d = 0, float eps = 0.f);
// h[m][n] += sum_s part[s][m][n], the splits added in order; with o16 (and
// olo) also the fp16 pair of the updated rows, as gemm()'s EPI_RESID; with ss
// (N a multiple of 256) the sums of squares of the new rows per 128 columns,
// ss[m][n / 128], for the next RMSNorm.
hipError_t part_resid(const float* part, int splits, int M, int N, float* h, void* o16, void* olo, hipStream_t s,
                      float* ss = nullptr);

// The 256 x 256-tile fp16 GEMM that gemm() picks for large prefix builds,
// callable for any M (N a multiple of 256, K of 64); same epilogues.
// bn: tile width, 256, 128 (N a multiple of 128) or (EPI_STORE, N a multiple of
// 192) 192; gemm() picks it.
hipError_t gemm_big(int epi, const void* u, const void* W, int M, int N, int K, void* out, int ldo, hipStream_t s,
                    int bn = 256);
// Split-K form of it (1 <= splits <= K/64): part[s][m][n] = the s-th of `splits`
// equal ranges of K steps of sum_k u[m][k] W[n][k]; part holds splits * M * N
// floats.  part_resid adds them to the residual.
hipError_t gemm_big_part(const void* u, const void* W, int M, int N, int K, int splits, float* part, hipStream_t s);

// Decode GEMV with the preceding RMSNorm fused (fp16, M <= 16), on the fp16
// copy x = hhi (+ hlo, its rounding error, when non-NULL) of the residual rows:
// y[m] = (W x[m]) / sqrt(mean(hhi[m]^2) + eps), followed by the epilogue as in
// gemm() (o16 / olo as there).  W carries the RMSNorm gain (folded at packing).
hipError_t gemv_rmsnorm(int ct, int epi, const void* hhi, float eps, const void* W, int M, int N, int K, void* out,
                        int ldo, hipStream_t s, const void* hlo = nullptr, void* o16 = nullptr,
                        void* olo = nullptr);

// Per row b: argmax over logits[b][0..n_bins) (lowest index on ties) -> out_tok[b*A+j],
// logits copied to out_logits[b][j] (if non-NULL); when feed, h[b] = bin_embed[t]
// with t the argmax or the clamped forced[b*A+j], and (if h16 is non-NULL, fp16
// compute only) h16[b] = the same row in fp16 and h16lo[b] (if non-NULL) = 0,
// its rounding error.
hipError_t argmax_feed(int ct, const float* logits, int ld_logits, const void* bin_embed, int B, int d, int n_bins,
                       int A, int j, int32_t* out_tok, float* out_logits, const int32_t* forced, float* h, int feed,
                       hipStream_t s, void* h16 = nullptr, void* h16lo = nullptr);

// u[m] = h[m] / sqrt(mean(h[m]^2) + eps), written in the compute type (the
// gain is folded into the weights that consume u).
// ulo (fp16 only, or NULL): the rounding error of u, so that u + ulo is the
// normalised row to about 22 significant bits.
hipError_t rmsnorm(int ct, const float* h, int M, int d, float eps, void* u, hipStream_t s, void* ulo = nullptr);
// h[m] += sum of the split-K partial sums part[s][m] (splits in order), then
// u[m] = fp16(h[m] / rms(h[m])) (fp16 compute; d <= 16384): part_resid and
// rmsnorm in one pass, u bitwise what rmsnorm gives.
hipError_t resid_norm(const float* part, int splits, int M, int d, float* h, float eps, void* u, hipStream_t s);

// out[i] = E[clamp(ids[i])] in the storage type.
hipError_t embed_rows(int st, const void* E, const int32_t* ids, int n, int d, int vocab, void* out,
                      hipStream_t s);

// h[i] = float(x[i]) for n rows of d (x in the storage type).
hipError_t ingest(int st, const void* x, int n, int d, float* h, hipStream_t s);
// The same per segment of a pass: its tokens come from input tokens src[s] ..
// (device array, one entry per segment of sg).
hipError_t ingest_segs(int st, const void* x, Segs sg, const int32_t* src, int d, float* h, hipStream_t s);

// Gate/up interleave of one layer: dst [2F][d] (compute type) from gate [F][d]
// and up [F][d] (storage type), each column k scaled by gain[k] (the RMSNorm
// gain folded into the weights).
hipError_t pack_gate_up(int st, int ct, const void* gate, const void* up, const float* gain, int F, int d, void* dst,
                        hipStream_t s);

// dst[n][k] = ct(src[n][k] * gain[k]) for a [rows][cols] matrix (gain == NULL:
// plain conversion; storage -> compute type; fp16 saturates).
hipError_t convert(int st, int ct, const void* src, size_t rows, int cols, const float* gain, void* dst,
                   hipStream_t s);

// tab[t][i] = (cos, sin)(t * theta^(-2i/dh)) for t < cap, i < dh/2 (computed in fp64).
hipError_t rope_table(float2* tab, int cap, int dh, float theta, hipStream_t s);

// Rotates the new tokens' keys and writes K/V into the slab of one layer.
// The QKV projection of a token pass with the K/V append in its epilogue: q
// columns stored fp32 at qkv[m][0..d) (ldo 3d), k rotated (RoPE at the token's
// position) and v written fp16 into the paged pools.  tok_base[m] = element
// offset of (page, head 0, slot) of token m in a layer's pool, tok_pos[m] its
// position (tok_tables).  Any M (head_dim 64 or 128, d a multiple of 256); the
// engine uses it where gemm_qkv_fusable(M, 3d, dh, d) holds, i.e. where gemm()
// would take the 256 x 256-tile GEMM for the projection.
struct KvEpi {
  const int64_t* tok_base = nullptr;
  const int32_t* tok_pos = nullptr;
  void* k = nullptr;  // fp16 pools of the layer
  void* v = nullptr;
  const float2* rope = nullptr;
  int d = 0, dh = 0;
};
bool gemm_qkv_fusable(int M, int N, int dh, int d);
hipError_t gemm_qkv_kv(const void* u, const void* W, int M, int K, float* qkv, const KvEpi& kv, hipStream_t s);
hipError_t tok_tables(Segs sg, KvPages kp, int H, int dh, int64_t* tok_base, int32_t* tok_pos, hipStream_t s);
hipError_t kv_append(int ct, const float* qkv, Segs sg, int H, int dh, KvPages kp, const float2* rope,
                     void* kslab, void* vslab, hipStream_t s);
// fp16 K/V append of a pass's n_tok tokens from the pass's token tables (tok_tables)
hipError_t kv_append_tab(const float* qkv, int n_tok, const int64_t* tok_base, const int32_t* tok_pos, int H, int dh,
                         const float2* rope, void* kslab, void* vslab, hipStream_t s);

// Causal attention of the pass's tokens over each row's slab (cache + new).
hipError_t attn_prefill(int ct, const float* qkv, Segs sg, int H, int dh, KvPages kp,
                        const float2* rope, const void* kslab, const void* vslab, void* o,
                        hipStream_t s);

// One query per row at position lens[b] + jpos: appends its K/V, attends over
// positions 0..lens[b]+jpos.  splits == 1: the output goes straight to o;
// otherwise the keys are cut into `splits` chunks whose partials (m, l, acc)
// go to `part` for attn_merge.  olo (fp16 only, or NULL): the rounding error of
// the fp16 output o, written by whichever of the two kernels writes o.
// The QKV projection's split-K partial sums (splits x [B][3d] floats) in place of
// qkv: the attention adds them in split order and divides row b by its rms
// from ss[b][0..nss) (sums of squares of the unnormalised residual per 128
// columns, width d; NULL: no scale), as part_store would.
struct QkvParts {
  const float* part = nullptr;
  int splits = 0;
  const float* ss = nullptr;
  int nss = 0;
  float eps = 0.f;
};
// order: NULL, or a permutation of the B rows (longest first, see len_order)
// in which their workgroups are dispatched; the results do not depend on it.
hipError_t attn_decode(int ct, const float* qkv, const int32_t* lens, int jpos, int B, int H, int dh,
                       int cap, KvPages kp, int splits, const float2* rope, void* kslab, void* vslab, float* part, void* o,
                       hipStream_t s, void* olo = nullptr, QkvParts qp = QkvParts{}, const int32_t* order = nullptr);
hipError_t attn_merge(int ct, const float* part, int B, int H, int dh, int splits, void* o,
                      hipStream_t s, void* olo = nullptr);

// h_last[row[s]] = h[off[s+1]-1] for each segment, and the same rows as fp16
// (saturating) into h_last16 when it is non-NULL, with their rounding error
// into h_last16lo when that is non-NULL too.
hipError_t gather_last(const float* h, Segs sg, int d, float* h_last, hipStream_t s, void* h_last16 = nullptr,
                       void* h_last16lo = nullptr);

// The whole greedy decode of a step in one persistent launch (fp16 compute,
// M <= 8 rows; see decode_fused.hip): head on the last committed position, then
// A - 1 times feed + all layers + head, with the outputs of argmax_feed.
// Pointers into the packed model (per-layer byte strides) and the context
// workspace; hp / op / ap are fp16 pairs laid out hi block then lo block
// ([2][M][width]); hl / hl_lo the pair of the last committed position (hl_lo
// after hl); part holds max(d/16, 1024) * 8 * 16 floats (enough for the
// split-K sums and for M*H*split_a attention partials of dh + 2 floats) and
// sync fused_sync_words(d, H) words.  The launch first clears sync with a kernel.
struct FusedDecode {
  const void *wqkv, *wo, *wgu, *wd, *whead, *bin_embed;  // matrices in fragment order (frag_pack)
  size_t s_qkv, s_o, s_gu, s_d;
  int L, d, H, dh, F, nbp, n_bins;
  float eps;
  int M, cap, A, split_o, split_d, split_a;
  const int32_t* lens;
  const float2* rope;
  void* kv;
  size_t slab_elems;
  const int32_t* pt;  // page table [M][ppr] of the context's K/V pages
  int ppr;
  float* h;
  void* hp;
  const void *hl, *hl_lo;
  float* qkv;
  void *op, *ap;
  float *logits, *part;
  unsigned* sync;
  unsigned* status;  // device view of a host-visible word, set to 1 when a barrier wait gives up (or NULL)
  int32_t* out_tok;
  float* out_logits;
  const int32_t* forced;
};
hipError_t decode_fused(const FusedDecode& f, int grid, hipStream_t s);
// Workgroups of the persistent decode on `device` (one per compute unit), 0 if
// it cannot be resident there.
int decode_fused_grid(int device, int dh);
int fused_sync_words(int d, int H);

// lens[b] += add[b] (device arrays), or, when `set`, lens[b] = add[b] for the
// rows with add[b] > 0 (a row-level rebuild leaves the other rows' lengths).
hipError_t update_lens(int32_t* lens, const int32_t* add, int B, int set, hipStream_t s);

// order[r] = the row of rank r by decreasing lens (ties by row index): a
// permutation of [0, B) computed on the device, so a captured decode graph
// follows the lengths of each replay.
hipError_t len_order(const int32_t* lens, int B, int32_t* order, hipStream_t s);

// Two-phase hashing for the action index (index.hip).  hash_segments: phase 1,
// seg_out[g] = HashFunc1 of bytes [g s, g s + s) of data (zero-padded past
// n_bytes), for g < ceil(n_bytes / s); s a multiple of 16 in [16, 65536], data
// 16-byte aligned.  hash_merge: phase 2, out[0] = HashFunc2 of seg[0..k) and
// n_bytes.  hash_page_keys: for each of B rows, keys[b][m] = HashFunc2 of the
// row's segments (starting at seg + seg_first[b]) covering its first
// (m + 1) page_bytes bytes, m < min(row_bytes[b] / page_bytes, max_pages)
// (device arrays; page_bytes a multiple of s).  Values pack the two 31-bit
// components (first base low).
hipError_t hash_segments(const void* data, uint64_t n_bytes, int s, uint64_t* seg_out, hipStream_t st);
hipError_t hash_merge(const uint64_t* seg, uint64_t k, uint64_t n_bytes, uint64_t* out, hipStream_t st);
hipError_t hash_page_keys(const uint64_t* seg, const int64_t* seg_first, const int64_t* row_bytes, int B,
                          int64_t page_bytes, int s, int max_pages, uint64_t* keys, hipStream_t st);

// The allocation-free variant's scratch: the device address, for `device`
// (which must be current), of the static array holding its segment hashes.
constexpr uint64_t INDEX_NOALLOC_MAX_SEGMENTS = 131072;
hipError_t index_noalloc_scratch(int device, uint64_t** ptr);

// Host tier (tier.hip): copies whole rows between the K/V page pools (pool =
// the context's K/V region, layer l's K at 2l * slab_layer bytes, V at
// (2l + 1) * slab_layer) plus the last hidden state (h_last fp32 [rows][d] and
// its fp16 pair h16 / h16lo) and host images at rows[i].host (a device-usable
// address of pinned host memory): after a 256-byte header, K/V
// [layer][K|V][head][len][dh] in the compute type (es bytes), then h_last [d]
// fp32 and the pair [d] + [d] fp16.  `rows` is a device array.
struct XferRow {
  int32_t row, len;
  void* host;
};
hipError_t rows_xfer(bool to_host, const XferRow* rows, int n_rows, int L, int H, int dh, int es, void* pool,
                     size_t slab_layer, const int32_t* pt, int ppr, float* h_last, void* h16, void* h16lo, int d,
                     hipStream_t s);

// Flow-matching action head (flow.hip), over the n_tok tokens of a pass (x and
// h of the pass's first token): flow_embed h[t] = W_in x[t] + tau w_t (W_in
// [d][a], w_t [d] in the storage type st); flow_update x[t] += dt W_out
// (h[t] / sqrt(mean(h[t]^2) + eps)) (W_out [a][d]).  1 <= a <= FLOW_MAX_ACTION_DIM.
constexpr int FLOW_MAX_ACTION_DIM = 256;
hipError_t flow_embed(int st, const float* x, const void* w_in, const void* w_t, float tau, int n_tok, int a, int d,
                      float* h, hipStream_t s);
hipError_t flow_update(int st, const float* h, const void* w_out, float eps, float dt, int n_tok, int a, int d,
                       float* x, hipStream_t s);

// Measured peaks (peaks.hip): a grid-stride copy of `bytes` (16-byte aligned
// pointers and size) from src to dst; a grid-stride read of src whose per-thread
// sums land in out[grid * 256]; `iters` rounds of fp16 MFMA chains per wave on
// register operands (all x; shape 0: 8 chains of 16x16x32, 1: 4 of 32x32x16,
// the same work), each thread's sum of its accumulators in out[grid * 256]
// (= 1024 x^2 iters while exact in fp32); mfma_loop_flops is the work of one
// such launch.  Not used by the decoder.
hipError_t stream_copy(const void* src, void* dst, size_t bytes, int grid, hipStream_t s);
hipError_t stream_read(const void* src, size_t bytes, float* out, int grid, hipStream_t s);
hipError_t mfma_loop(int shape, float x, int iters, float* out, int grid, hipStream_t s);
double mfma_loop_flops(int iters, int grid);

}  // namespace ams
