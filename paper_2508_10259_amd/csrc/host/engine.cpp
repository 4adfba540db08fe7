// Engine: weight packing, context set-up, the token forward pass (prefix
// build and observation extension) and the greedy decode loop, which is
// captured once per (n_actions, output buffers) into a HIP graph and replayed.
#include "engine.h"

#include <stdlib.h>

#include "../kernels/kernels.h"

namespace ams {

#define TRY(expr)                                                        \
  do {                                                                   \
    hipError_t e_ = (expr);                                              \
    if (e_ != hipSuccess) {                                              \
      err = std::string(#expr) + ": " + hipGetErrorString(e_);           \
      return e_;                                                         \
    }                                                                    \
  } while (0)

static const char* off(const void* p, size_t bytes) { return (const char*)p + bytes; }

// Decode runs its RMSNorms inside the projection GEMVs for fp16 compute and up
// to 8 rows (see norm_proj).
static bool fused_norm(const Ctx& c, int rows) { return c.model->ct == DT_F16 && rows <= 8; }

// Above 8 rows the fp16 decode GEMVs use the wide GEMM (128 weight rows per
// workgroup, activations staged in LDS) with split-K partial sums: at 16 rows
// of the 7B model it decodes 4% faster than the skinny GEMV with separate lo
// fragments.
static bool wide_decode(const Ctx& c, int rows, int N) {
  return c.model->ct == DT_F16 && rows > 8 && rows <= 64 && N % 128 == 0;
}

// On the wide path the RMSNorm of a projection input needs no kernel of its
// own once a residual reduction has run: it leaves the unnormalised fp16 pair
// of h in (u, hlo) and its sums of squares per 128 columns, and the
// projection's reduction divides its rows by rms.
// Up to 16 rows the wide GEMM reduces its split-K partial sums in each tile's
// last split instead of a separate kernel: measured on the 7B decoder at 16
// rows, O 14.0 -> 12.6 us, down 23.6 -> 22.1 us, gate|up 41.0 -> 39.7 us; at 64
// rows the O and down projections' 32 tiles would reduce on 32 CUs, 1-5 us
// slower per projection.
static bool wide_fused_reduce(int rows) { return rows <= 16; }

static bool merge_norm(const Ctx& c, int rows) {
  const Cfg& m = c.model->cfg;
  return wide_decode(c, rows, m.d_model) && m.d_model % 256 == 0 && m.d_ffn % 256 == 0 && bins_padded(m) % 256 == 0;
}

// The persistent decode (decode_fused) serves fp16 compute up to 8 rows when
// the shapes fit its tiling and its 32-bit buffer offsets; AMS_FUSED=0 turns it
// off (the per-kernel decode then runs).
static bool fused_applies(const Ctx& c) {
  const char* e = getenv("AMS_FUSED");
  if (e && e[0] == '0') return false;
  const Cfg& m = c.model->cfg;
  const int B = c.lay.batch;
  if (c.model->ct != DT_F16 || B > FUSED_MAX_ROWS) return false;
  if (m.head_dim != 64 && m.head_dim != 128) return false;
  if (m.d_model % 128 != 0 || m.d_ffn % 128 != 0 || bins_padded(m) % 16 != 0) return false;
  return c.lay.slab_layer < ((size_t)1 << 31) && (size_t)B * 3 * m.d_model * 4 < ((size_t)1 << 31) &&
         (size_t)B * m.d_ffn * 4 < ((size_t)1 << 31);
}

hipError_t model_pack(Model& m, const ams_weights_view& w, hipStream_t s, std::string& err) {
  // bf16 weights become fp16 in the packed copy: exact for |w| >= 2^-14, an
  // fp16 subnormal (absolute error <= 2^-25) below; fp32 models are copied.
  // Each RMSNorm gain is folded into the columns of the matrices that read the
  // normalised vector: W u = (W diag(g)) (h / rms(h)).
  const Cfg& c = m.cfg;
  const size_t es = elem_size(c), d = c.d_model, F = c.d_ffn;
  const size_t dde = d * d * es;
  const int st = m.st, ct = m.ct;
  for (int l = 0; l < c.n_layers; ++l) {
    char* qkv = (char*)m.wqkv(l);
    const float* ga = w.g_attn + (size_t)l * d;
    const float* gf = w.g_ffn + (size_t)l * d;
    TRY(convert(st, ct, off(w.w_q, l * dde), d, (int)d, ga, qkv, s));
    TRY(convert(st, ct, off(w.w_k, l * dde), d, (int)d, ga, qkv + dde, s));
    TRY(convert(st, ct, off(w.w_v, l * dde), d, (int)d, ga, qkv + 2 * dde, s));
    TRY(convert(st, ct, off(w.w_o, l * dde), d, (int)d, nullptr, (void*)m.wo(l), s));
    TRY(pack_gate_up(st, ct, off(w.w_gate, l * F * d * es), off(w.w_up, l * F * d * es), gf, (int)F, (int)d,
                     (void*)m.wgu(l), s));
    TRY(convert(st, ct, off(w.w_down, l * d * F * es), d, (int)F, nullptr, (void*)m.wd(l), s));
  }
  TRY(hipMemsetAsync(m.ws + m.lay.head_bins, 0, (size_t)bins_padded(c) * d * es, s));
  TRY(convert(st, ct, w.head_bins, c.n_bins, (int)d, w.g_final, m.ws + m.lay.head_bins, s));
  TRY(convert(st, ct, off(w.embed, (size_t)(c.vocab - c.n_bins) * d * es), c.n_bins, (int)d, nullptr,
              m.ws + m.lay.bin_embed, s));
  if (ct == DT_F16) {  // the decode passes' copies in MFMA fragment order
    for (int l = 0; l < c.n_layers; ++l) {
      TRY(frag_pack(m.wqkv(l), 3 * (int)d, (int)d, (void*)m.fqkv(l), s));
      TRY(frag_pack(m.wo(l), (int)d, (int)d, (void*)m.fo(l), s));
      TRY(frag_pack(m.wgu(l), 2 * (int)F, (int)d, (void*)m.fgu(l), s));
      TRY(frag_pack(m.wd(l), (int)d, (int)F, (void*)m.fd(l), s));
    }
    TRY(frag_pack(m.head_bins(), bins_padded(c), (int)d, (void*)m.fhead(), s));
  }
  return hipSuccess;
}

// The page table to the device, rows without pages pointing at page 0.
static hipError_t upload_pages(Ctx& c, hipStream_t s) {
  c.pt_dev_host.resize(c.pt_host.size());
  for (size_t i = 0; i < c.pt_host.size(); ++i) c.pt_dev_host[i] = c.pt_host[i] < 0 ? 0 : c.pt_host[i];
  return hipMemcpyAsync(c.pt(), c.pt_dev_host.data(), c.pt_dev_host.size() * 4, hipMemcpyHostToDevice, s);
}

hipError_t ctx_init(Ctx& c, std::string& err) {
  const Cfg& m = c.model->cfg;
  TRY(hipStreamCreateWithFlags(&c.capture_stream, hipStreamNonBlocking));
  void* st = nullptr;
  TRY(hipHostMalloc(&st, 256, hipHostMallocMapped));
  c.status_host = (volatile unsigned*)st;
  *c.status_host = 0u;
  TRY(hipHostGetDevicePointer((void**)&c.status_dev, st, 0));
  hipStream_t s = c.capture_stream;
  TRY(rope_table(c.rope(), c.lay.capacity, m.head_dim, m.rope_theta, s));
  TRY(hipMemsetAsync(c.ws + c.lay.h_last, 0, c.lay.part - c.lay.h_last, s));
  TRY(hipMemsetAsync(c.ws + c.lay.lens, 0, c.lay.total - c.lay.lens, s));
  // fixed pages: row b's page i is b * ppr + i; pooled: no row holds a page yet
  // (-1 on the host; the device table holds page 0 there, never read before a build)
  c.pt_host.assign((size_t)c.lay.batch * c.lay.ppr, -1);
  if (c.pooled) c.pool.init(c.lay.n_pages);
  else
    for (size_t i = 0; i < c.pt_host.size(); ++i) c.pt_host[i] = (int32_t)i;
  TRY(upload_pages(c, s));
  TRY(hipStreamSynchronize(s));
  c.splits = decode_splits(c.lay.batch, m.n_heads, c.lay.capacity);
  c.meta_host.assign(c.lay.meta_ints, 0);
  c.fused_grid = fused_applies(c) ? decode_fused_grid(c.model->device, m.head_dim) : 0;
  if (c.fused_grid > 0) {
    c.split_o = fused_split(m, m.d_model, c.fused_grid);
    c.split_d = fused_split(m, m.d_ffn, c.fused_grid);
    c.split_a = fused_split_attn(m, c.lay.batch, c.lay.capacity, c.fused_grid);
  }
  return hipSuccess;
}

void ctx_release(Ctx& c) {
  if (!c.graphs.empty()) hipDeviceSynchronize();
  for (auto& kv : c.graphs) hipGraphExecDestroy(kv.second);
  c.graphs.clear();
  c.graph_lru.clear();
  if (c.capture_stream) hipStreamDestroy(c.capture_stream);
  c.capture_stream = nullptr;
  if (c.status_host) hipHostFree((void*)c.status_host);
  c.status_host = nullptr;
  c.status_dev = nullptr;
}

void ctx_release_rows(Ctx& c, const int32_t* rows, int n_rows) {
  if (!c.pooled) return;
  // the released rows' entries become -1 on the host; the device keeps the stale
  // ones, which no kernel reads before those rows are rebuilt
  release_row_pages(c.pool, c.pt_host, c.lay.ppr, rows, n_rows);
}

int ctx_build_rows(Ctx& c, const void* prefix, const int32_t* rows, int n_rows, const int32_t* lens, hipStream_t s,
                   std::string& err) {
  const Cfg& m = c.model->cfg;
  const int B = c.lay.batch, ppr = c.lay.ppr;
  const size_t tb = (size_t)m.d_model * elem_size(m);
  std::vector<int32_t> counts(B, 0), start(B, 0), src(B, 0), lens_set(B, 0);
  if (!c.pooled) {
    for (int i = 0; i < n_rows; ++i) counts[rows[i]] = lens_set[rows[i]] = lens[i];
    return ctx_forward_tokens(c, prefix, counts.data(), start.data(), 1, s, err) == hipSuccess ? (int)S_OK
                                                                                                : (int)S_EHIP;
  }
  std::vector<int32_t> share(n_rows, 0), first(n_rows, 0);
  size_t tok = 0;
  for (int i = 0; i < n_rows; ++i) {
    first[i] = (int32_t)tok;
    tok += lens[i];
    share[i] = c.lay.share ? shareable_pages(lens[i]) : 0;
  }
  c.keys_host.assign((size_t)n_rows * ppr, 0);
  if (c.lay.share) {  // page keys: Algorithm 1 over each row's input bytes up to every page end
    const int sg = c.lay.key_seg;
    const size_t nseg = tok * tb / sg;
    uint64_t* seg = (uint64_t*)(c.ws + c.lay.hk_seg);
    uint64_t* keys = (uint64_t*)(c.ws + c.lay.hk_keys);
    int64_t* hk = (int64_t*)(c.ws + c.lay.hk_rows);
    c.hk_rows_host.assign(2 * (size_t)n_rows, 0);
    for (int i = 0; i < n_rows; ++i) {
      c.hk_rows_host[i] = (int64_t)first[i] * (int64_t)(tb / sg);
      c.hk_rows_host[n_rows + i] = (int64_t)lens[i] * (int64_t)tb;
    }
    if (hash_segments(prefix, tok * tb, sg, seg, s) != hipSuccess ||
        hipMemcpyAsync(hk, c.hk_rows_host.data(), c.hk_rows_host.size() * 8, hipMemcpyHostToDevice, s) !=
            hipSuccess ||
        hash_page_keys(seg, hk, hk + n_rows, n_rows, (int64_t)64 * tb, sg, ppr, keys, s) != hipSuccess ||
        hipMemcpyAsync(c.keys_host.data(), keys, c.keys_host.size() * 8, hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess) {
      err = "page keys of the prefix failed";
      return S_EHIP;
    }
    (void)nseg;
  }
  std::vector<int32_t> st;
  if (int r = plan_row_pages(c.pool, c.pt_host, ppr, rows, n_rows, share.data(), c.keys_host.data(), ppr,
                             c.lay.share, st, err))
    return r;
  if (upload_pages(c, s) != hipSuccess) {
    err = "page table upload failed";
    return S_EHIP;
  }
  for (int i = 0; i < n_rows; ++i) {
    const int b = rows[i];
    start[b] = st[i];
    counts[b] = lens[i] - st[i];
    src[b] = first[i] + st[i];
    lens_set[b] = lens[i];
  }
  return ctx_forward_tokens(c, prefix, counts.data(), start.data(), 1, s, err, src.data(), lens_set.data()) ==
                 hipSuccess
             ? (int)S_OK
             : (int)S_EHIP;
}

static int rows_xfer_enqueue(Ctx& c, bool to_host, const int32_t* rows, int n_rows, const int32_t* lens,
                             void* const* host_dev, hipStream_t s, std::string& err) {
  const Cfg& m = c.model->cfg;
  c.xfer_host.resize(n_rows);
  for (int i = 0; i < n_rows; ++i) c.xfer_host[i] = XferRow{rows[i], lens[i], host_dev[i]};
  XferRow* xd = (XferRow*)(c.ws + c.lay.xfer);
  if (hipMemcpyAsync(xd, c.xfer_host.data(), n_rows * sizeof(XferRow), hipMemcpyHostToDevice, s) != hipSuccess ||
      rows_xfer(to_host, xd, n_rows, m.n_layers, m.n_heads, m.head_dim, (int)(c.model->ct == DT_F16 ? 2 : 4),
                c.ws + c.lay.kv, c.lay.slab_layer, c.pt(), c.lay.ppr, c.h_last(), c.h_last16(), c.h_last16lo(),
                m.d_model, s) != hipSuccess) {
    err = to_host ? "offload to host memory failed" : "reload from host memory failed";
    return S_EHIP;
  }
  return S_OK;
}

int ctx_offload_rows(Ctx& c, const int32_t* rows, int n_rows, const int32_t* lens, void* const* host_dev,
                     hipStream_t s, std::string& err) {
  if (int r = rows_xfer_enqueue(c, true, rows, n_rows, lens, host_dev, s, err)) return r;
  // the pages go back to the pool now; work enqueued later on the same stream,
  // which may reuse them, runs after the copies
  ctx_release_rows(c, rows, n_rows);
  return S_OK;
}

int ctx_reload_rows(Ctx& c, const int32_t* rows, int n_rows, const int32_t* lens, void* const* host_dev,
                    hipStream_t s, std::string& err) {
  const int B = c.lay.batch;
  if (c.pooled) {
    std::vector<int32_t> share(n_rows, 0), st;
    if (int r = plan_row_pages(c.pool, c.pt_host, c.lay.ppr, rows, n_rows, share.data(), nullptr, 0, false, st, err))
      return r;
    if (upload_pages(c, s) != hipSuccess) {
      err = "page table upload failed";
      return S_EHIP;
    }
  }
  if (int r = rows_xfer_enqueue(c, false, rows, n_rows, lens, host_dev, s, err)) return r;
  // the rows' device lengths: set mode of the length update over a [B] array
  std::vector<int32_t>& h = c.meta_host;
  std::fill(h.begin(), h.end(), 0);
  for (int i = 0; i < n_rows; ++i) h[4 * B + 1 + rows[i]] = lens[i];
  int32_t* md = c.meta();
  if (hipMemcpyAsync(md, h.data(), h.size() * sizeof(int32_t), hipMemcpyHostToDevice, s) != hipSuccess ||
      update_lens(c.lens(), md + 4 * B + 1, B, 1, s) != hipSuccess) {
    err = "length update failed";
    return S_EHIP;
  }
  return S_OK;
}

int ctx_absorb_status(Ctx& c, std::string& err) {
  if (!c.status_host) return S_OK;
  const unsigned w = *c.status_host;
  if (w) *c.status_host = 0u;
  return c.book.absorb_async_error(w, err);
}

// The K/V append rides in the QKV projection's epilogue where that GEMM takes
// 256 x 256 tiles (7B build: 201 us per layer of k_kv_append and the fp32 k/v
// columns of qkv saved).
static bool kv_fusable(const Ctx& c, int M) {
  const Cfg& m = c.model->cfg;
  return c.model->ct == DT_F16 && gemm_qkv_fusable(M, 3 * m.d_model, m.head_dim, m.d_model);
}

// h += x W^T over the M tokens of a token pass (K inputs per token).  At
// medium token counts in fp16 the 256 x 256-tile GEMM splits K and a reduction
// adds the partial sums in split order; that reduction also leaves the next
// RMSNorm's output in u (normed = true), which saves the norm its own pass
// over h (7B, 1,024-token extension: 6.4 us per norm).
static hipError_t tokens_resid(Ctx& c, const void* x, const void* W, int M, int K, hipStream_t s, bool& normed) {
  const Model& md = *c.model;
  const int d = md.cfg.d_model;
  const int splits = md.ct == DT_F16 ? prefill_ksplit(M, d, K) : 1;
  normed = false;
  if (splits > 1) {
    hipError_t e = gemm_big_part(x, W, M, d, K, splits, c.kpart(), s);
    if (e == hipSuccess) e = resid_norm(c.kpart(), splits, M, d, c.h(), md.cfg.rms_eps, c.u(), s);
    normed = e == hipSuccess;
    return e;
  }
  return gemm(md.ct, EPI_RESID, x, W, M, d, K, c.h(), d, s);
}

// One decoder layer over the M tokens of a token pass; u_ready: u already holds
// RMSNorm(h) (left by the previous residual reduction), and on return whether
// it holds the norm of this layer's output; tables: the pass's token tables
// are in the workspace (fp16: every token pass); kv_fused: the QKV projection
// appends K/V itself from them.
static hipError_t layer_tokens(Ctx& c, int l, int M, const Segs& sg, hipStream_t s, std::string& err, bool& u_ready,
                               bool tables, bool kv_fused) {
  const Model& md = *c.model;
  const Cfg& m = md.cfg;
  const int d = m.d_model, F = m.d_ffn, dt = md.ct;
  if (!u_ready) TRY(rmsnorm(dt, c.h(), M, d, m.rms_eps, c.u(), s));
  if (kv_fused) {  // the QKV GEMM's epilogue appends K/V (the token tables are the pass's)
    KvEpi kv{(const int64_t*)(c.ws + c.lay.tok_base), (const int32_t*)(c.ws + c.lay.tok_pos), c.kslab(l), c.vslab(l),
             c.rope(), d, m.head_dim};
    TRY(gemm_qkv_kv(c.u(), md.wqkv(l), M, d, c.qkv(), kv, s));
  } else {
    TRY(gemm(dt, EPI_STORE, c.u(), md.wqkv(l), M, 3 * d, d, c.qkv(), 3 * d, s));
    if (tables)  // each token's slot from the pass's tables (7B batch-64 extension: 19.05 -> 18.92 ms per step)
      TRY(kv_append_tab(c.qkv(), M, (const int64_t*)(c.ws + c.lay.tok_base), (const int32_t*)(c.ws + c.lay.tok_pos),
                        m.n_heads, m.head_dim, c.rope(), c.kslab(l), c.vslab(l), s));
    else
      TRY(kv_append(dt, c.qkv(), sg, m.n_heads, m.head_dim, c.pages(), c.rope(), c.kslab(l), c.vslab(l), s));
  }
  TRY(attn_prefill(dt, c.qkv(), sg, m.n_heads, m.head_dim, c.pages(), c.rope(), c.kslab(l), c.vslab(l), c.o(),
                   s));
  TRY(tokens_resid(c, c.o(), md.wo(l), M, d, s, u_ready));
  if (!u_ready) TRY(rmsnorm(dt, c.h(), M, d, m.rms_eps, c.u(), s));
  TRY(gemm(dt, EPI_SWIGLU, c.u(), md.wgu(l), M, 2 * F, d, c.a(), F, s));
  TRY(tokens_resid(c, c.a(), md.wd(l), M, F, s, u_ready));
  return hipSuccess;
}

hipError_t ctx_forward_tokens(Ctx& c, const void* x, const int32_t* counts, const int32_t* start, int set_lens,
                              hipStream_t s, std::string& err, const int32_t* src, const int32_t* lens_set) {
  const Cfg& m = c.model->cfg;
  const int B = c.lay.batch;
  const size_t es = elem_size(m), d = m.d_model;
  Plan p = plan_passes(B, counts, start, c.lay.pass_tokens);
  // meta layout: row[B] pos[B] off[2B+1] lensv[B] src[B] (src per segment: its first input token)
  std::vector<int32_t>& h = c.meta_host;
  std::fill(h.begin(), h.end(), 0);
  std::copy(p.row.begin(), p.row.end(), h.begin());
  std::copy(p.pos.begin(), p.pos.end(), h.begin() + B);
  std::copy(p.off.begin(), p.off.end(), h.begin() + 2 * B);
  for (int b = 0; b < B; ++b) h[4 * B + 1 + b] = lens_set ? lens_set[b] : counts[b];
  if (src)
    for (size_t i = 0; i < p.row.size(); ++i) h[5 * B + 1 + i] = src[p.row[i]];
  const std::vector<int32_t> ord = pass_orders(p, counts);
  std::copy(ord.begin(), ord.end(), h.begin() + 6 * B + 1);
  int32_t* md = c.meta();
  TRY(hipMemcpyAsync(md, h.data(), h.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  for (size_t pi = 0; pi < p.passes.size(); ++pi) {
    const Pass& ps = p.passes[pi];
    Segs sg{md + ps.seg_begin, md + B + ps.seg_begin, md + 2 * B + ps.seg_begin + (int)pi, ps.n_seg, ps.n_tok,
            ps.max_len, ps.max_end, md + 6 * B + 1 + ps.seg_begin};
    if (src)  // the rows' tokens to process start at their own places in x
      TRY(ingest_segs(c.model->st, x, sg, md + 5 * B + 1 + ps.seg_begin, (int)d, c.h(), s));
    else
      TRY(ingest(c.model->st, (const char*)x + (size_t)ps.tok_src * d * es, ps.n_tok, (int)d, c.h(), s));
    bool u_ready = false;
    const bool tabs = c.model->ct == DT_F16, kvf = kv_fusable(c, ps.n_tok);
    if (tabs)
      TRY(tok_tables(sg, c.pages(), m.n_heads, m.head_dim, (int64_t*)(c.ws + c.lay.tok_base),
                     (int32_t*)(c.ws + c.lay.tok_pos), s));
    for (int l = 0; l < m.n_layers; ++l)
      if (layer_tokens(c, l, ps.n_tok, sg, s, err, u_ready, tabs, kvf) != hipSuccess) return hipErrorLaunchFailure;
    const bool f16 = c.model->ct == DT_F16;  // the fp16 pair of h_last feeds fused-RMSNorm heads
    TRY(gather_last(c.h(), sg, (int)d, c.h_last(), s, f16 ? c.h_last16() : nullptr, f16 ? c.h_last16lo() : nullptr));
  }
  TRY(update_lens(c.lens(), md + 4 * B + 1, B, set_lens, s));
  return hipSuccess;
}

hipError_t ctx_flow(Ctx& c, const FlowHeadView& fh, float* x, float tau0, int n_steps, hipStream_t s,
                    std::string& err) {
  const Cfg& m = c.model->cfg;
  const int B = c.lay.batch, T = fh.n_tokens, a = fh.a, d = m.d_model;
  if (n_steps <= 0) return hipSuccess;
  std::vector<int32_t> counts(B, T), start(c.book.len.begin(), c.book.len.end());
  Plan p = plan_passes(B, counts.data(), start.data(), c.lay.pass_tokens);
  std::vector<int32_t>& h = c.meta_host;
  std::fill(h.begin(), h.end(), 0);
  std::copy(p.row.begin(), p.row.end(), h.begin());
  std::copy(p.pos.begin(), p.pos.end(), h.begin() + B);
  std::copy(p.off.begin(), p.off.end(), h.begin() + 2 * B);
  const std::vector<int32_t> ord = pass_orders(p, counts.data());
  std::copy(ord.begin(), ord.end(), h.begin() + 6 * B + 1);
  int32_t* md = c.meta();
  TRY(hipMemcpyAsync(md, h.data(), h.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  const float dt = (1.0f - tau0) / (float)n_steps;
  for (int k = 0; k < n_steps; ++k) {
    const float tau = tau0 + (float)k * dt;
    for (size_t pi = 0; pi < p.passes.size(); ++pi) {
      const Pass& ps = p.passes[pi];
      Segs sg{md + ps.seg_begin, md + B + ps.seg_begin, md + 2 * B + ps.seg_begin + (int)pi, ps.n_seg, ps.n_tok,
              ps.max_len, ps.max_end, md + 6 * B + 1 + ps.seg_begin};
      float* xp = x + (size_t)ps.tok_src * a;  // every row brings T tokens: the pass's first token
      TRY(flow_embed(c.model->st, xp, fh.w_in, fh.w_t, tau, ps.n_tok, a, d, c.h(), s));
      const bool tabs = c.model->ct == DT_F16;
      if (tabs)
        TRY(tok_tables(sg, c.pages(), m.n_heads, m.head_dim, (int64_t*)(c.ws + c.lay.tok_base),
                       (int32_t*)(c.ws + c.lay.tok_pos), s));
      bool u_ready = false;
      for (int l = 0; l < m.n_layers; ++l)
        if (layer_tokens(c, l, ps.n_tok, sg, s, err, u_ready, tabs, false) != hipSuccess) return hipErrorLaunchFailure;
      TRY(flow_update(c.model->st, c.h(), fh.w_out, m.rms_eps, dt, ps.n_tok, a, d, xp, s));
    }
  }
  return hipSuccess;
}

// Decode-pass GEMV inputs are fp16 pairs (hi + lo, lo the rounding error of
// hi) in fp16 compute, so the action tokens' own products see their inputs to
// about 22 significant bits; the MFMA count doubles at most, the weight stream
// (the bound) does not change.
//
// Rows is a view of the per-row buffers from row r0 on (n rows): every decode
// kernel addresses rows relative to the pointers it is given.
struct Rows {
  int r0, n;
  size_t ces;  // bytes of a compute-type element
  const Ctx* c;
  char* at(size_t off, size_t row_bytes) const { return c->ws + off + (size_t)r0 * row_bytes; }
  float* h() const { return (float*)at(c->lay.h, c->model->cfg.d_model * 4); }
  void* u() const { return at(c->lay.u, c->model->cfg.d_model * ces); }
  float* qkv() const { return (float*)at(c->lay.qkv, 3 * c->model->cfg.d_model * 4); }
  void* o() const { return at(c->lay.o, c->model->cfg.d_model * ces); }
  void* a() const { return at(c->lay.a, c->model->cfg.d_ffn * ces); }
  float* h_last() const { return (float*)at(c->lay.h_last, c->model->cfg.d_model * 4); }
  void* h_last16() const { return at(c->lay.h_last16, c->model->cfg.d_model * 2); }
  void* h_last16lo() const { return at(c->lay.h_last16lo, c->model->cfg.d_model * 2); }
  void* hlo() const { return at(c->lay.hlo, c->model->cfg.d_model * 2); }
  void* olo() const { return at(c->lay.olo, c->model->cfg.d_model * 2); }
  void* alo() const { return at(c->lay.alo, c->model->cfg.d_ffn * 2); }
  float* logits() const { return (float*)at(c->lay.logits, bins_padded(c->model->cfg) * 4); }
  float* ss() const { return (float*)at(c->lay.ss, (size_t)(c->model->cfg.d_model / 128) * 4); }
  int32_t* lens() const { return (int32_t*)at(c->lay.lens, 4); }
  int32_t* order() const { return (int32_t*)at(c->lay.order, 4); }
  float* part() const {
    const Cfg& m = c->model->cfg;
    return (float*)at(c->lay.part, (size_t)m.n_heads * c->splits * (m.head_dim + 2) * 4);
  }
  // the layer's page pools; the rows' page tables start at row r0
  void* kslab(int l) const { return c->kslab(l); }
  void* vslab(int l) const { return c->vslab(l); }
  KvPages pages() const { return KvPages{c->pt() + (size_t)r0 * c->lay.ppr, c->lay.ppr}; }
};

// Projection of a normalised input.  Up to 8 fp16 rows run the GEMV with the
// RMSNorm fused, reading the fp16 pair of the residual rows (hhi, hlo) that
// their producers (residual GEMV epilogue, feed, gather of the last prefix
// token) write beside h; otherwise rmsnorm writes the pair u + hlo from h
// first (the fused copies are unused then, so hlo serves as u's lo part) --
// except on the wide path with ss, where (u, hlo) already hold the
// unnormalised pair and the reduction divides by rms (merge_norm).
static hipError_t norm_proj(const Rows& g, int epi, const float* h, const void* hhi, const void* hlo, const void* W,
                            const void* Wf, int N, int K, void* out, int ldo, void* olo, hipStream_t s,
                            std::string& err, const float* ss = nullptr, QkvParts* defer = nullptr) {
  const Model& md = *g.c->model;
  const float eps = md.cfg.rms_eps;
  if (fused_norm(*g.c, g.n)) {
    TRY(gemv_rmsnorm(md.ct, epi, hhi, eps, W, g.n, N, K, out, ldo, s, hlo, nullptr, olo));
  } else {
    void* ulo = md.ct == DT_F16 ? g.hlo() : nullptr;
    const bool wide = wide_decode(*g.c, g.n, N);
    if (!(wide && ss)) {
      ss = nullptr;
      TRY(rmsnorm(md.ct, h, g.n, K, eps, g.u(), s, ulo));
    }
    if (wide) {  // partial sums of 128-row tiles, then the epilogue
      // When the attention adds the partial sums, every split costs each of its
      // workgroups another read of its q, k, v slices: two splits measured
      // best on the 7B decoder at 64 rows (decode 47.2 / 45.9 / 45.0 / 44.8 ms
      // per step at 8 / 4 / 5 / 2 splits).
      const int splits = defer ? std::max(1, std::min(2, K >> 7)) : decode_wsplit(N, K);
      if (!defer && wide_fused_reduce(g.n)) {
        TRY(gemm_wide_reduce(epi, g.u(), ulo, Wf, g.n, N, K, splits, g.c->kpart(), g.c->wcnt(), out, olo, ldo, nullptr,
                             nullptr, nullptr, nullptr, ss, eps, s));
      } else {
        TRY(gemm_wide(g.u(), ulo, Wf, g.n, N, K, splits, g.c->kpart(), s));
        if (defer) {  // the consumer adds the partial sums itself
          *defer = QkvParts{g.c->kpart(), splits, ss, K / 128, eps};
        } else if (epi == EPI_SWIGLU) {
          TRY(part_swiglu(g.c->kpart(), splits, g.n, N, out, olo, s, ss, K, eps));
        } else {
          TRY(part_store(g.c->kpart(), splits, g.n, N, (float*)out, s, ss, K, eps));
        }
      }
    } else {
      TRY(gemm(md.ct, epi, g.u(), W, g.n, N, K, out, ldo, s, ulo, nullptr, olo));
    }
  }
  return hipSuccess;
}

// h += W x for the decode rows (x = the pair x + xlo in fp16 compute), writing
// the fp16 pair of the new rows to (hhi, hlo) when given.  Narrow projections
// split K over more workgroups and add the partial sums in a reduction kernel;
// on the wide path with ss that reduction also leaves the unnormalised pair in
// (u, hlo) and the sums of squares in ss for the next projection.
static hipError_t resid_proj(const Rows& g, const void* x, const void* xlo, const void* W, const void* Wf, int K,
                             void* hhi, void* hlo, hipStream_t s, float* ss = nullptr) {
  const Ctx& c = *g.c;
  const Model& md = *c.model;
  const int d = md.cfg.d_model;
  if (wide_decode(c, g.n, d)) {
    const int splits = decode_wsplit(d, K);
    void* o16 = ss ? g.u() : hhi;
    void* olo = ss ? g.hlo() : hlo;
    if (wide_fused_reduce(g.n))
      return gemm_wide_reduce(EPI_RESID, x, xlo, Wf, g.n, d, K, splits, c.kpart(), c.wcnt(), nullptr, nullptr, 0,
                              g.h(), o16, olo, ss, nullptr, 0.f, s);
    hipError_t e = gemm_wide(x, xlo, Wf, g.n, d, K, splits, c.kpart(), s);
    if (e == hipSuccess) e = part_resid(c.kpart(), splits, g.n, d, g.h(), o16, olo, s, ss);
    return e;
  }
  const int splits = md.ct == DT_F16 ? decode_ksplit(d, K) : 1;
  if (splits > 1) {
    hipError_t e = gemm_part(x, xlo, W, g.n, d, K, splits, c.kpart(), s);
    if (e == hipSuccess) e = part_resid(c.kpart(), splits, g.n, d, g.h(), hhi, hlo, s);
    return e;
  }
  return gemm(md.ct, EPI_RESID, x, W, g.n, d, K, g.h(), d, s, xlo, hhi, hlo);
}

// One decoder layer for the rows' fed-back tokens at positions lens[b] + jpos.
static hipError_t layer_decode(const Rows& g, int l, int jpos, hipStream_t s, std::string& err) {
  const Ctx& c = *g.c;
  const Model& md = *c.model;
  const Cfg& m = md.cfg;
  const int d = m.d_model, F = m.d_ffn, dt = md.ct, B = g.n;
  const bool f16 = dt == DT_F16, fused = fused_norm(c, B);
  void* hhi = fused ? g.u() : nullptr;   // fp16 pair of h (fused path)
  void* hlo = fused ? g.hlo() : nullptr;
  void* olo = f16 ? g.olo() : nullptr;   // lo parts of the attention and SwiGLU outputs
  void* alo = f16 ? g.alo() : nullptr;
  // sums of squares of h from the previous residual reduction (from layer 1 on)
  float* ss = merge_norm(c, B) ? g.ss() : nullptr;
  // on the wide path the attention adds the QKV projection's partial sums itself
  QkvParts qp{};
  if (norm_proj(g, EPI_STORE, g.h(), hhi, hlo, md.wqkv(l), md.fqkv(l), 3 * d, d, g.qkv(), 3 * d, nullptr, s, err,
                l > 0 ? ss : nullptr, &qp) != hipSuccess)
    return hipErrorLaunchFailure;
  TRY(attn_decode(dt, g.qkv(), g.lens(), jpos, B, m.n_heads, m.head_dim, c.lay.capacity, g.pages(), c.splits, c.rope(),
                  g.kslab(l), g.vslab(l), g.part(), g.o(), s, olo, qp, B > 1 ? g.order() : nullptr));
  if (c.splits > 1) TRY(attn_merge(dt, g.part(), B, m.n_heads, m.head_dim, c.splits, g.o(), s, olo));
  TRY(resid_proj(g, g.o(), olo, md.wo(l), md.fo(l), d, hhi, hlo, s, ss));
  if (norm_proj(g, EPI_SWIGLU, g.h(), hhi, hlo, md.wgu(l), md.fgu(l), 2 * F, d, g.a(), F, alo, s, err, ss) != hipSuccess)
    return hipErrorLaunchFailure;
  TRY(resid_proj(g, g.a(), alo, md.wd(l), md.fd(l), F, hhi, hlo, s, ss));
  return hipSuccess;
}

// Action head for decode position j: final RMSNorm + bin logits (the
// projection GEMV over the padded head rows), then argmax/outputs/feed.
// tok / logits / forced point at the group's first row.
static hipError_t head(const Rows& g, const float* hin, const void* hhi, const void* hlo, int A, int j, int32_t* tok,
                       float* logits, const int32_t* forced, hipStream_t s, std::string& err,
                       const float* ss = nullptr) {
  const Model& md = *g.c->model;
  const Cfg& m = md.cfg;
  const int d = m.d_model, nbp = bins_padded(m);
  const bool fused = fused_norm(*g.c, g.n);
  if (norm_proj(g, EPI_STORE, hin, hhi, hlo, md.head_bins(), md.fhead(), nbp, d, g.logits(), nbp, nullptr, s, err, ss) !=
      hipSuccess)
    return hipErrorLaunchFailure;
  TRY(argmax_feed(md.ct, g.logits(), nbp, md.bin_embed(), g.n, d, m.n_bins, A, j, tok, logits, forced, g.h(),
                  j + 1 < A, s, fused ? g.u() : nullptr, fused ? g.hlo() : nullptr));
  return hipSuccess;
}

static hipError_t decode_rows(const Rows& g, int A, int32_t* tok, float* logits, const int32_t* forced, hipStream_t s,
                              std::string& err) {
  const Cfg& m = g.c->model->cfg;
  const bool fused = fused_norm(*g.c, g.n);
  int32_t* gt = tok + (size_t)g.r0 * A;
  float* gl = logits ? logits + (size_t)g.r0 * A * m.n_bins : nullptr;
  const int32_t* gf = forced ? forced + (size_t)g.r0 * A : nullptr;
  // the rows longest first for the decode attention's dispatch (one order per
  // step: every pass adds one position to every row)
  if (g.n > 1 && A > 1) TRY(len_order(g.lens(), g.n, g.order(), s));
  if (head(g, g.h_last(), fused ? g.h_last16() : nullptr, fused ? g.h_last16lo() : nullptr, A, 0, gt, gl, gf, s,
           err) != hipSuccess)
    return hipErrorLaunchFailure;
  for (int j = 1; j < A; ++j) {
    for (int l = 0; l < m.n_layers; ++l)
      if (layer_decode(g, l, j - 1, s, err) != hipSuccess) return hipErrorLaunchFailure;
    // after the last layer's residual reduction: its sums of squares, when kept
    const float* ss = merge_norm(*g.c, g.n) && m.n_layers > 0 ? g.ss() : nullptr;
    if (head(g, g.h(), fused ? g.u() : nullptr, fused ? g.hlo() : nullptr, A, j, gt, gl, gf, s, err, ss) !=
        hipSuccess)
      return hipErrorLaunchFailure;
  }
  return hipSuccess;
}

// The greedy loop of a step as one persistent launch.
static hipError_t enqueue_fused(Ctx& c, int A, int32_t* tok, float* logits, const int32_t* forced, hipStream_t s,
                                std::string& err) {
  const Model& md = *c.model;
  const Cfg& m = md.cfg;
  FusedDecode f{};
  f.wqkv = md.fqkv(0); f.s_qkv = md.lay.per_layer_qkv;  // fragment-ordered copies
  f.wo = md.fo(0); f.s_o = md.lay.per_layer_o;
  f.wgu = md.fgu(0); f.s_gu = md.lay.per_layer_gu;
  f.wd = md.fd(0); f.s_d = md.lay.per_layer_d;
  f.whead = md.fhead();
  f.bin_embed = md.bin_embed();
  f.L = m.n_layers; f.d = m.d_model; f.H = m.n_heads; f.dh = m.head_dim; f.F = m.d_ffn;
  f.nbp = bins_padded(m); f.n_bins = m.n_bins; f.eps = m.rms_eps;
  f.M = c.lay.batch; f.cap = c.lay.capacity; f.A = A;
  f.split_o = c.split_o; f.split_d = c.split_d; f.split_a = c.split_a;
  f.lens = c.lens(); f.rope = c.rope();
  f.kv = c.ws + c.lay.kv; f.slab_elems = c.lay.slab_layer / 2;
  f.pt = c.pt(); f.ppr = c.lay.ppr;
  f.h = c.h(); f.hp = c.ws + c.lay.fx_hp;
  f.hl = c.h_last16(); f.hl_lo = c.h_last16lo();
  f.qkv = c.qkv(); f.op = c.ws + c.lay.fx_op; f.ap = c.ws + c.lay.fx_ap;
  f.logits = c.logits(); f.part = (float*)(c.ws + c.lay.fx_part); f.sync = (unsigned*)(c.ws + c.lay.fx_sync);
  f.status = c.status_dev;
  f.out_tok = tok; f.out_logits = logits; f.forced = forced;
  TRY(decode_fused(f, c.fused_grid, s));
  return hipSuccess;
}

// The greedy loop of a step over all rows.
static hipError_t enqueue_decode(Ctx& c, int A, int32_t* tok, float* logits, const int32_t* forced, hipStream_t s,
                                 std::string& err) {
  if (c.fused_grid > 0) return enqueue_fused(c, A, tok, logits, forced, s, err);
  const size_t ces = c.model->ct == DT_F16 ? 2 : 4;
  return decode_rows(Rows{0, c.lay.batch, ces, &c}, A, tok, logits, forced, s, err);
}

static bool graphs_enabled() {
  const char* e = getenv("AMS_GRAPH");
  return !(e && e[0] == '0');
}

hipError_t ctx_decode(Ctx& c, int A, int32_t* tok, float* logits, const int32_t* forced, hipStream_t s,
                      std::string& err) {
  if (!graphs_enabled()) return enqueue_decode(c, A, tok, logits, forced, s, err);
  GraphKey key{A, tok, logits, forced};
  auto it = c.graphs.find(key);
  if (it == c.graphs.end()) {
    hipStream_t cs = c.capture_stream;
    TRY(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal));
    hipError_t e = enqueue_decode(c, A, tok, logits, forced, cs, err);
    hipGraph_t g = nullptr;
    hipError_t e2 = hipStreamEndCapture(cs, &g);
    if (e != hipSuccess) {
      if (g) hipGraphDestroy(g);
      return e;
    }
    if (e2 != hipSuccess) {
      err = std::string("hipStreamEndCapture: ") + hipGetErrorString(e2);
      return e2;
    }
    hipGraphExec_t ex = nullptr;
    hipError_t e3 = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    hipGraphDestroy(g);
    if (e3 != hipSuccess) {
      err = std::string("hipGraphInstantiate: ") + hipGetErrorString(e3);
      return e3;
    }
    if (c.graph_lru.size() >= 8) {
      TRY(hipStreamSynchronize(s));  // the evicted graph may still be running on s
      auto old = c.graphs.find(c.graph_lru.front());
      if (old != c.graphs.end()) {
        hipGraphExecDestroy(old->second);
        c.graphs.erase(old);
      }
      c.graph_lru.erase(c.graph_lru.begin());
    }
    it = c.graphs.emplace(key, ex).first;
    c.graph_lru.push_back(key);
  }
  TRY(hipGraphLaunch(it->second, s));
  return hipSuccess;
}

}  // namespace ams
