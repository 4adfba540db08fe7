// Host-only bookkeeping of the cached-context decoder: configuration checks,
// device workspace layouts, the per-row length book (commit / rollback /
// invalidate) and the planner that packs ragged rows into forward passes.
// No HIP dependency: the CPU tests compile this header with a plain C++
// compiler and sanitizers.
#pragma once

#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <cmath>
#include <string>
#include <unordered_map>
#include <vector>

#include "fused_limits.h"

namespace ams {

enum Status { S_OK = 0, S_EINVAL = -1, S_ESTATE = -2, S_ECAPACITY = -3, S_ENODEV = -4, S_EHIP = -5, S_ENOMEM = -6 };

struct Cfg {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, n_bins;
  float rms_eps, rope_theta;
  int32_t dtype;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Segment size of the page keys: the largest power of two <= 4096 dividing the
// bytes of one token's input, so that rows and pages start on segment bounds.
inline int page_key_segment(size_t token_bytes) {
  int s = 4096;
  while (s > 16 && token_bytes % s) s >>= 1;
  return s;
}


inline int check_cfg(const Cfg& c, std::string& err) {
  auto bad = [&](const char* m) { err = m; return (int)S_EINVAL; };
  if (c.n_layers < 1 || c.n_layers > 1024) return bad("n_layers must be in [1, 1024]");
  if (c.head_dim != 64 && c.head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c.n_heads < 1 || (int64_t)c.n_heads * c.head_dim != c.d_model) return bad("d_model must equal n_heads * head_dim");
  if (c.d_model % 128 != 0 || c.d_model > 16384) return bad("d_model must be a multiple of 128 and <= 16384");
  if (c.d_ffn < 128 || c.d_ffn % 128 != 0 || c.d_ffn > 65536) return bad("d_ffn must be a multiple of 128 in [128, 65536]");
  if (c.n_bins < 1 || c.n_bins > 1024) return bad("n_bins must be in [1, 1024]");
  if (c.vocab < c.n_bins || c.vocab > (1 << 24)) return bad("vocab must be in [n_bins, 2^24]");
  if (!(c.rms_eps > 0.f) || !std::isfinite(c.rms_eps)) return bad("rms_eps must be finite and > 0");
  if (!(c.rope_theta > 1.f) || !std::isfinite(c.rope_theta)) return bad("rope_theta must be finite and > 1");
  if (c.dtype != 0 && c.dtype != 1) return bad("dtype must be AMS_F32 (0) or AMS_BF16 (1)");
  return S_OK;
}

inline size_t elem_size(const Cfg& c) { return c.dtype == 0 ? 4 : 2; }

// Rows of the packed action head, padded with zero rows to a multiple of 64
// so the head runs through the same GEMV/GEMM kernels as the projections.
inline int bins_padded(const Cfg& c) { return (c.n_bins + 63) / 64 * 64; }

// Model workspace: packed weights (RMSNorm gains folded in), the bin rows of
// the head and of the embedding table.  Offsets in bytes from the workspace base.
struct ModelLayout {
  size_t wqkv, wo, wgu, wd, head_bins, bin_embed, total;
  size_t per_layer_qkv, per_layer_o, per_layer_gu, per_layer_d;  // bytes per layer
  // fp16 compute: a second copy of the decode-pass matrices in MFMA fragment
  // order (frag_pack), same per-layer strides; 0 / unused for fp32 models
  size_t fqkv, fo, fgu, fd, fhead;
};

inline ModelLayout model_layout(const Cfg& c) {
  const size_t es = elem_size(c), d = c.d_model, F = c.d_ffn, L = c.n_layers;
  ModelLayout m{};
  m.per_layer_qkv = 3 * d * d * es;
  m.per_layer_o = d * d * es;
  m.per_layer_gu = 2 * F * d * es;
  m.per_layer_d = d * F * es;
  size_t o = 0;
  m.wqkv = o; o = align256(o + L * m.per_layer_qkv);
  m.wo = o; o = align256(o + L * m.per_layer_o);
  m.wgu = o; o = align256(o + L * m.per_layer_gu);
  m.wd = o; o = align256(o + L * m.per_layer_d);
  m.head_bins = o; o = align256(o + (size_t)bins_padded(c) * d * es);
  m.bin_embed = o; o = align256(o + (size_t)c.n_bins * d * es);
  if (es == 2) {
    m.fqkv = o; o = align256(o + L * m.per_layer_qkv);
    m.fo = o; o = align256(o + L * m.per_layer_o);
    m.fgu = o; o = align256(o + L * m.per_layer_gu);
    m.fd = o; o = align256(o + L * m.per_layer_d);
    m.fhead = o; o = align256(o + (size_t)bins_padded(c) * d * es);
  }
  m.total = o;
  return m;
}

// Context workspace: the K/V slab, activations of one forward pass, and
// small device-side tables.
struct CtxLayout {
  int batch, capacity, pass_tokens, max_splits;
  int ppr;            // K/V pages per row (capacity / 64)
  int n_pages;        // pages in each layer's K (and V) pool
  size_t slab_layer;  // bytes of K (or V) for one layer: n_pages pages of 64 positions
  size_t kv, h, u, qkv, o, a, h_last, h_last16, h_last16lo, hlo, olo, alo, kpart, part, logits, rope, lens, meta, total;
  size_t order;  // the rows by decreasing length [B] int32 (decode attention dispatch order)
  size_t tok_base, tok_pos;  // a token pass's pool offsets [T] int64 and positions [T] int32 (K/V append)
  size_t ss;  // decode rows' sums of squares per 128 residual columns [B][d/128]
  size_t wcnt;  // arrival counters of the wide decode GEMM's weight tiles (zero between launches)
  // persistent decode (fp16, up to 8 rows): fp16 pairs [2][B][width] of h, the
  // attention output and the SwiGLU output, split-K partials, sync words
  size_t fx_hp, fx_op, fx_ap, fx_part, fx_sync;
  size_t meta_ints;
  size_t pt;  // page table [batch][ppr] int32
  // shared prefix pages: segment hashes of a build's input, page keys [batch][ppr]
  // and per-row [segment offset, input bytes] (int64) of the hashed rows
  bool share;
  int key_seg;  // segment size of the page keys (bytes)
  size_t hk_seg, hk_keys, hk_rows;
  size_t xfer;  // host-tier transfer descriptors [batch] (16 bytes each)
};

// Bytes of the host image of a row of `len` positions (see the host tier).
inline size_t row_host_bytes(const Cfg& c, int len) {
  return 256 + (size_t)2 * c.n_layers * len * c.d_model * elem_size(c) + (size_t)c.d_model * (4 + 2 + 2);
}

inline int default_pass_tokens(int batch, int capacity) {
  const int64_t bc = (int64_t)batch * capacity;
  int t = (int)std::min<int64_t>(bc, 32768);
  return std::max(t, capacity);
}

// K splits of a residual decode GEMV with N output rows and K inputs: when its
// 16-row strips are fewer than one per CU (256), the K range is cut so that
// strips x splits reaches about 256 workgroups, keeping at least 8 chunks of
// 128 per split (a reduction kernel, ~3 us, then adds the partial sums into h,
// which shorter ranges do not repay).
inline int decode_ksplit(int N, int K) {
  const int strips = N / 16;
  if (strips >= 256) return 1;
  const int s = std::min(256 / std::max(strips, 1), (K / 128) / 8);
  return std::max(1, s);
}

// K splits of a wide decode GEMM (more than 8 rows; 128 weight rows per
// workgroup, at least 4 chunks of 128 per split, at most 16 splits).  The time
// model is the rounds of workgroups per CU over the work per workgroup,
// ceil(tiles * S / 256) / S on the 256 CUs; every further split also adds
// partial sums and staging, so the smallest S within 5% of the model's minimum
// is taken.  On the 7B shapes at 16 and 64 rows this is the measured best of
// S = 1..8 (QKV 8, gate|up 4, O and down 8); counts that leave the last round
// of workgroups mostly empty lose to both neighbours.
inline int decode_wsplit(int N, int K) {
  const int tiles = std::max(N / 128, 1), smax = std::max(1, std::min(16, (K / 128) / 4));
  auto t = [&](int s) { return (double)((tiles * s + 255) / 256) / s; };
  double best = t(1);
  for (int s = 2; s <= smax; ++s) best = std::min(best, t(s));
  int s = 1;
  while (t(s) > 1.05 * best) ++s;
  return s;
}

// Persistent decode (one launch per step) applies up to this many rows.
constexpr int FUSED_MAX_ROWS = 8;
// Split-K units of its O and down projections: at most this many.
inline size_t fused_part_units(const Cfg& c) { return std::max<size_t>(c.d_model / 16, 1024); }
// K splits of a residual projection (d/16 strips over K/128 chunks) in the
// persistent decode on `grid` workgroups: a unit's weights should stay within
// 32 KB (the two weight batches a workgroup loads while it waits at the
// barrier before the phase), as long as there are workgroups to spare.  On the
// 12-layer d=1024 decoder at 8 rows the down projection (128 KB per strip)
// measured 8.2 / 6.1 / 5.0 us per phase split 1 / 2 / 4 ways, while splitting
// the O projection (32 KB per strip) in two cost 1.1 us more.
inline int fused_split(const Cfg& c, int K, int grid) {
  const int strips = c.d_model / 16, nch = K / 128;
  if (strips >= grid) return 1;
  const size_t unit_bytes = (size_t)16 * K * 2;
  int s = (int)std::min<size_t>((unit_bytes + 32767) / 32768, (size_t)(grid / std::max(strips, 1)));
  s = std::max(1, std::min({s, nch, FUSED_MAX_SPLIT}));
  while (s > 1 && (size_t)strips * s > fused_part_units(c)) --s;
  return s;
}

// Key splits of its attention.  A split's keys take one round of its 8 waves
// when they number at most 8 waves x (5 or 8 iterations) x (64 / (head_dim / 8))
// keys per iteration (320 at head_dim 64, 256 at 128).  Merging splits costs a memory round trip, so more splits than
// that are taken only when (row, head) items would leave at least 3 in 4
// workgroups idle (then up to 8).  Partials stay within the split-K buffer.
inline int fused_split_attn(const Cfg& c, int rows, int capacity, int grid) {
  const int items = rows * c.n_heads, round = 8 * (c.head_dim == 64 ? 5 : 8) * (64 / (c.head_dim / 8));
  const int need = (capacity + round - 1) / round;  // splits for one round each
  const int spare = grid / std::max(items, 1);      // splits the idle workgroups allow
  int s = std::max(need, spare >= 4 ? std::min(spare, 8) : 1);
  s = std::max(1, std::min(s, FUSED_MAX_ATTN_SPLIT));
  while (s > 1 && (size_t)items * s * (c.head_dim + 2) > fused_part_units(c) * 8 * 16) --s;
  return s;
}

// K splits of a residual projection of a token pass (fp16; N = d_model output
// rows, K inputs): the 256 x 256-tile GEMM takes token counts whose tiles number
// 160 or more unsplit; below that, when N is a multiple of 256 and the pass has
// more than 64 tokens, its K steps (of 64) are cut so that tiles x splits
// reaches about 256 workgroups, each keeping at least 8 K steps.
inline int prefill_ksplit(int M, int N, int K) {
  if (M <= 64 || N % 256 != 0 || K % 64 != 0) return 1;
  const int tiles = (N / 256) * ((M + 255) / 256);
  if (tiles >= 160) return 1;
  return std::max(1, std::min((256 + tiles - 1) / tiles, (K / 64) / 8));
}

// Floats of split-K partial sums the token passes of a context need (at most
// pass_tokens tokens per pass; the O projection has K = d, the down projection
// K = F).
inline size_t prefill_part_floats(const Cfg& c, int pass_tokens) {
  size_t best = 0;
  const int d = c.d_model, F = c.d_ffn;
  for (int M = 65; M <= pass_tokens; M = M < 256 ? 256 : M + 256) {
    const int m = std::min(M, pass_tokens);
    const int s = std::max(prefill_ksplit(m, d, d), prefill_ksplit(m, d, F));
    if (s > 1) best = std::max(best, (size_t)s * m * d);
    if ((d / 256) * ((m + 255) / 256) >= 160) break;
  }
  return best;
}

inline int check_ctx_args(const Cfg& c, int batch, int capacity, int pass_tokens, std::string& err) {
  if (batch < 1 || batch > 1024) { err = "batch must be in [1, 1024]"; return S_EINVAL; }
  if (capacity < 64 || capacity % 64 != 0 || capacity > (1 << 20)) {
    err = "capacity must be a multiple of 64 in [64, 2^20]";
    return S_EINVAL;
  }
  if (pass_tokens != 0 && (pass_tokens < capacity || pass_tokens > (1 << 22))) {
    err = "max_pass_tokens must be 0 or in [capacity, 2^22]";
    return S_EINVAL;
  }
  (void)c;
  return S_OK;
}

// n_pages: K/V pages per layer pool (0: batch * capacity / 64, a page for every
// position of every row); share: rows may share prefix pages (hash scratch).
inline CtxLayout ctx_layout(const Cfg& c, int batch, int capacity, int pass_tokens, int n_pages = 0,
                            bool share = false) {
  CtxLayout x{};
  const size_t es = elem_size(c), d = c.d_model, F = c.d_ffn, L = c.n_layers, B = batch;
  x.batch = batch;
  x.capacity = capacity;
  x.pass_tokens = pass_tokens ? pass_tokens : default_pass_tokens(batch, capacity);
  x.max_splits = capacity / 64;
  x.ppr = capacity / 64;
  x.n_pages = n_pages > 0 ? n_pages : batch * x.ppr;
  const size_t T = std::max<size_t>(x.pass_tokens, B);
  x.slab_layer = (size_t)x.n_pages * 64 * d * es;
  size_t o = 0;
  x.kv = o; o = align256(o + 2 * L * x.slab_layer);
  x.h = o; o = align256(o + T * d * 4);
  x.u = o; o = align256(o + T * d * es);
  x.qkv = o; o = align256(o + T * 3 * d * 4);
  x.o = o; o = align256(o + T * d * es);
  x.a = o; o = align256(o + T * F * es);
  x.h_last = o; o = align256(o + B * d * 4);
  // decode-pass fp16 pairs (hi, lo = rounding error of hi): hi of h lives in u,
  // hi of the attention / SwiGLU outputs in o / a; the lo parts here
  x.h_last16 = o; o = align256(o + B * d * 2);
  x.h_last16lo = o; o = align256(o + B * d * 2);
  x.hlo = o; o = align256(o + B * d * 2);
  x.olo = o; o = align256(o + B * d * 2);
  x.alo = o; o = align256(o + B * F * 2);
  // split-K partial sums (fp16 compute): the decode GEMVs' (the narrow residual
  // projections at up to 8 rows, every projection above 8 rows) and the token
  // passes' residual projections at medium token counts
  size_t kp = 0;
  const size_t ks = std::max(decode_ksplit((int)d, (int)d), decode_ksplit((int)d, (int)F));
  if (ks > 1) kp = ks * B * d;
  if (batch > 8 && batch <= 64) {
    const size_t NB = bins_padded(c);
    kp = std::max({kp, decode_wsplit(3 * (int)d, (int)d) * B * 3 * d, decode_wsplit((int)d, (int)d) * B * d,
                   decode_wsplit(2 * (int)F, (int)d) * B * 2 * F, decode_wsplit((int)d, (int)F) * B * d,
                   decode_wsplit((int)NB, (int)d) * B * NB});
  }
  if (es == 2) kp = std::max(kp, prefill_part_floats(c, (int)x.pass_tokens));
  x.kpart = o; o = align256(o + kp * 4);
  x.part = o; o = align256(o + B * (size_t)c.n_heads * x.max_splits * (c.head_dim + 2) * 4);
  x.logits = o; o = align256(o + B * (size_t)bins_padded(c) * 4);
  x.ss = o; o = align256(o + B * (size_t)(d / 128 + 1) * 4);
  x.rope = o; o = align256(o + (size_t)capacity * (c.head_dim / 2) * 8);
  x.lens = o; o = align256(o + B * 4);
  x.order = o; o = align256(o + B * 4);
  x.tok_base = o; o = align256(o + T * 8);
  x.tok_pos = o; o = align256(o + T * 4);
  // pass metadata of one call: row[B], pos[B], off[2B+1], lens staging[B], src[B],
  // order[B] (each pass's segments by decreasing pos + len, indices local to the pass)
  x.meta_ints = 7 * B + 1;
  x.meta = o; o = align256(o + x.meta_ints * 4);
  const bool fx = batch <= FUSED_MAX_ROWS && es == 2;
  x.fx_hp = o; o = align256(o + (fx ? 2 * B * d * 2 : 0));
  x.fx_op = o; o = align256(o + (fx ? 2 * B * d * 2 : 0));
  x.fx_ap = o; o = align256(o + (fx ? 2 * B * F * 2 : 0));
  x.fx_part = o; o = align256(o + (fx ? fused_part_units(c) * 8 * 16 * 4 : 0));
  x.fx_sync = o; o = align256(o + (fx ? (size_t)(32 * 64 + std::max<size_t>(d / 16, 8 * c.n_heads)) * 4 : 0));
  x.pt = o; o = align256(o + B * (size_t)x.ppr * 4);
  x.share = share;
  x.key_seg = page_key_segment(d * es);
  const size_t max_segs = share ? B * (size_t)capacity * (d * es / x.key_seg) : 0;
  x.hk_seg = o; o = align256(o + max_segs * 8);
  x.hk_keys = o; o = align256(o + (share ? B * (size_t)x.ppr * 8 : 0));
  x.hk_rows = o; o = align256(o + (share ? 2 * B * 8 : 0));
  x.xfer = o; o = align256(o + B * 16);
  x.wcnt = o; o = align256(o + std::max({3 * d, 2 * F, (size_t)bins_padded(c), d}) / 128 * 4);
  x.total = o;
  return x;
}

// ---------------------------------------------------------------------------
// length book: the host-side truth of each row's committed length

enum CtxState { EMPTY = 0, READY = 1, INVALID = 2, OFFLOADED = 3 };  // OFFLOADED: rows only

// Each row has its own state (EMPTY until first built, READY, INVALID after a
// row-level or whole-context invalidate); the context is READY when every row
// is, EMPTY while no row has been built, INVALID otherwise.  Only a READY
// context steps: a row that an exception handler invalidated must be rebuilt
// (alone, with the other rows' contexts untouched) before the batch steps on.
struct RowBook {
  int batch = 0, capacity = 0;
  int state = EMPTY;
  std::vector<int32_t> len;
  std::vector<int8_t> row_state;

  void init(int b, int cap) {
    batch = b;
    capacity = cap;
    state = EMPTY;
    len.assign(b, 0);
    row_state.assign(b, (int8_t)EMPTY);
  }

  void refresh_state() {  // (an offloaded row makes the context INVALID until reloaded)
    bool all_ready = true, all_empty = true;
    for (int b = 0; b < batch; ++b) {
      all_ready = all_ready && row_state[b] == READY;
      all_empty = all_empty && row_state[b] == EMPTY;
    }
    state = all_ready ? READY : all_empty ? EMPTY : INVALID;
  }

  int check_build(const int32_t* lens, std::string& err) const {
    if (!lens) { err = "lens is NULL"; return S_EINVAL; }
    for (int b = 0; b < batch; ++b) {
      if (lens[b] < 1) { err = "prefix length must be >= 1 (row " + std::to_string(b) + ")"; return S_EINVAL; }
      if (lens[b] > capacity) { err = "prefix longer than capacity (row " + std::to_string(b) + ")"; return S_ECAPACITY; }
    }
    return S_OK;
  }

  // rows: n strictly increasing row indices in [0, batch); lens[i]: new prefix
  // length of rows[i].
  int check_rows(const int32_t* rows, int n, std::string& err) const {
    if (!rows || n < 1 || n > batch) { err = "rows must list 1..batch row indices"; return S_EINVAL; }
    for (int i = 0; i < n; ++i) {
      if (rows[i] < 0 || rows[i] >= batch) { err = "row index out of range"; return S_EINVAL; }
      if (i && rows[i] <= rows[i - 1]) { err = "row indices must be strictly increasing"; return S_EINVAL; }
    }
    return S_OK;
  }

  int check_build_rows(const int32_t* rows, int n, const int32_t* lens, std::string& err) const {
    if (int s = check_rows(rows, n, err)) return s;
    if (!lens) { err = "lens is NULL"; return S_EINVAL; }
    for (int i = 0; i < n; ++i) {
      if (lens[i] < 1) { err = "prefix length must be >= 1 (row " + std::to_string(rows[i]) + ")"; return S_EINVAL; }
      if (lens[i] > capacity) {
        err = "prefix longer than capacity (row " + std::to_string(rows[i]) + ")";
        return S_ECAPACITY;
      }
    }
    return S_OK;
  }

  // new tokens only (no action decode): every row READY, len + n <= capacity
  int check_append(const int32_t* new_lens, std::string& err) const {
    if (state != READY) { err = state == EMPTY ? "context was never built" : "context (or a row of it) is invalidated"; return S_ESTATE; }
    if (!new_lens) { err = "new_lens is NULL"; return S_EINVAL; }
    for (int b = 0; b < batch; ++b) {
      if (new_lens[b] < 0) { err = "negative new length (row " + std::to_string(b) + ")"; return S_EINVAL; }
      if ((int64_t)len[b] + new_lens[b] > capacity) {
        err = "row " + std::to_string(b) + " would exceed capacity";
        return S_ECAPACITY;
      }
    }
    return S_OK;
  }

  int check_step(const int32_t* new_lens, int n_actions, std::string& err) const {
    if (state != READY) { err = state == EMPTY ? "context was never built" : "context (or a row of it) is invalidated"; return S_ESTATE; }
    if (n_actions < 1 || n_actions > capacity) { err = "n_actions must be in [1, capacity]"; return S_EINVAL; }
    for (int b = 0; b < batch; ++b) {
      const int64_t n = new_lens ? new_lens[b] : 0;
      if (n < 0) { err = "negative new length (row " + std::to_string(b) + ")"; return S_EINVAL; }
      if ((int64_t)len[b] + n + n_actions - 1 > capacity) {
        err = "row " + std::to_string(b) + " would exceed capacity";
        return S_ECAPACITY;
      }
    }
    return S_OK;
  }

  void commit_build(const int32_t* lens) {
    for (int b = 0; b < batch; ++b) {
      len[b] = lens[b];
      row_state[b] = READY;
    }
    state = READY;
  }
  void commit_build_rows(const int32_t* rows, int n, const int32_t* lens) {
    for (int i = 0; i < n; ++i) {
      len[rows[i]] = lens[i];
      row_state[rows[i]] = READY;
    }
    refresh_state();
  }
  void commit_new(const int32_t* new_lens) {
    if (!new_lens) return;
    for (int b = 0; b < batch; ++b) len[b] += new_lens[b];
  }
  void invalidate() {
    std::fill(len.begin(), len.end(), 0);
    std::fill(row_state.begin(), row_state.end(), (int8_t)INVALID);
    state = INVALID;
  }
  void invalidate_rows(const int32_t* rows, int n) {
    for (int i = 0; i < n; ++i) {
      len[rows[i]] = 0;
      row_state[rows[i]] = INVALID;
    }
    refresh_state();
  }
  // rows whose contexts moved to host memory: not steppable until reloaded
  // (length 0 meanwhile); every listed row must be READY
  int check_offload(const int32_t* rows, int n, std::string& err) const {
    if (int s = check_rows(rows, n, err)) return s;
    for (int i = 0; i < n; ++i)
      if (row_state[rows[i]] != READY) {
        err = "row " + std::to_string(rows[i]) + " holds no context to offload";
        return S_ESTATE;
      }
    return S_OK;
  }
  void offload_rows(const int32_t* rows, int n) {
    for (int i = 0; i < n; ++i) {
      len[rows[i]] = 0;
      row_state[rows[i]] = OFFLOADED;
    }
    refresh_state();
  }
  // a row may be reloaded unless it holds a context (READY)
  int check_reload(const int32_t* rows, int n, std::string& err) const {
    if (int s = check_rows(rows, n, err)) return s;
    for (int i = 0; i < n; ++i)
      if (row_state[rows[i]] == READY) {
        err = "row " + std::to_string(rows[i]) + " holds a context (invalidate or offload it first)";
        return S_ESTATE;
      }
    return S_OK;
  }

  // An error that a kernel reported asynchronously (the persistent decode's
  // status word: nonzero once a barrier wait gave up) is taken in by the next
  // call on the context: the context becomes INVALID and the call fails with
  // S_EHIP.  A zero word changes nothing.
  int absorb_async_error(unsigned word, std::string& err) {
    if (word == 0) return S_OK;
    invalidate();
    err = "an earlier action decode gave up waiting for its workgroups (not all resident at once); "
          "its tokens read -1 and the context was invalidated";
    return S_EHIP;
  }
};

// ---------------------------------------------------------------------------
// K/V page pool with shared prefix pages (paper section 3.2.3, Virtual Action):
// every page of a context has a reference count; a page holding a row's input
// up to its end can be published under its key (the two-phase hash of that
// input prefix, Algorithm 1), and a later row whose input agrees up to the same
// page end references that page instead of computing and storing its own.
// Attaching increments the count, invalidating a row decrements the counts of
// its pages, and a page whose count reaches zero leaves the index and returns
// to the free list.

struct PagePool {
  std::vector<int32_t> refs;
  std::vector<uint64_t> key;        // published key of a page (valid when indexed[p])
  std::vector<uint8_t> indexed;
  std::vector<int32_t> free_pages;  // stack; the lowest free page on top
  std::unordered_map<uint64_t, int32_t> index;

  void init(int n) {
    refs.assign(n, 0);
    key.assign(n, 0);
    indexed.assign(n, 0);
    free_pages.resize(n);
    for (int i = 0; i < n; ++i) free_pages[i] = n - 1 - i;
    index.clear();
  }
  int n_pages() const { return (int)refs.size(); }
  int in_use() const { return n_pages() - (int)free_pages.size(); }
  int alloc() {  // a fresh page with one reference, -1 when none is free
    if (free_pages.empty()) return -1;
    const int p = free_pages.back();
    free_pages.pop_back();
    refs[p] = 1;
    return p;
  }
  void retain(int p) { ++refs[p]; }
  void release(int p) {
    if (p < 0 || refs[p] <= 0) return;
    if (--refs[p] == 0) {
      if (indexed[p]) {
        auto it = index.find(key[p]);
        if (it != index.end() && it->second == p) index.erase(it);
        indexed[p] = 0;
      }
      free_pages.push_back(p);
    }
  }
  int lookup(uint64_t k) const {
    auto it = index.find(k);
    return it == index.end() ? -1 : it->second;
  }
  void publish(int p, uint64_t k) {
    key[p] = k;
    indexed[p] = 1;
    index[k] = p;
  }
};

// Pages of rows about to be built.  Each listed row (in order) first releases
// the pages it held, then takes, for its leading full pages that do not hold its
// last token (i < share[i_row], keys[i_row][i]), the published page of the same
// key when there is one (the row starts computing after the run of pages it
// could attach), else a fresh page that it publishes; its remaining ppr pages
// are fresh.  Writes the rows' page-table rows into pt ([batch][ppr]) and the
// first position each row computes into start[i_row].  Fails with S_ECAPACITY,
// pool and pt unchanged, when the pool runs out of free pages.
inline int plan_row_pages(PagePool& pool, std::vector<int32_t>& pt, int ppr, const int32_t* rows, int n_rows,
                          const int32_t* share, const uint64_t* keys, int keys_stride, bool sharing,
                          std::vector<int32_t>& start, std::string& err) {
  PagePool saved = pool;
  std::vector<int32_t> saved_pt = pt;
  for (int i = 0; i < n_rows; ++i)
    for (int j = 0; j < ppr; ++j) {
      int32_t& e = pt[(size_t)rows[i] * ppr + j];
      if (e >= 0) pool.release(e);
      e = -1;
    }
  start.assign(n_rows, 0);
  for (int i = 0; i < n_rows; ++i) {
    int32_t* row = &pt[(size_t)rows[i] * ppr];
    int attached = 0;
    for (int j = 0; j < ppr; ++j) {
      const bool shareable = sharing && j < share[i];
      if (shareable && j == attached) {
        const uint64_t k = keys[(size_t)i * keys_stride + j];
        const int p = pool.lookup(k);
        if (p >= 0) {
          pool.retain(p);
          row[j] = p;
          ++attached;
          continue;
        }
      }
      const int p = pool.alloc();
      if (p < 0) {
        pool = saved;
        pt = saved_pt;
        err = "the context's K/V page pool has no free page left (row " + std::to_string(rows[i]) + ")";
        return S_ECAPACITY;
      }
      row[j] = p;
      if (shareable) pool.publish(p, keys[(size_t)i * keys_stride + j]);
    }
    start[i] = attached * 64;
  }
  return S_OK;
}

// Releases the pages of the listed rows (their page-table entries become -1).
inline void release_row_pages(PagePool& pool, std::vector<int32_t>& pt, int ppr, const int32_t* rows, int n_rows) {
  for (int i = 0; i < n_rows; ++i)
    for (int j = 0; j < ppr; ++j) {
      int32_t& e = pt[(size_t)rows[i] * ppr + j];
      if (e >= 0) pool.release(e);
      e = -1;
    }
}

// Pages of a row that may be shared: the full 64-position pages before the one
// holding its last token (that token's hidden state must be computed).
inline int shareable_pages(int len) { return (len - 1) / 64; }

// ---------------------------------------------------------------------------
// Eviction plan of the layered store (paper sections 3.2.2 and 3.2.3, Auto
// Eviction): to free `need` pages, the resident unpinned rows are taken in
// increasing (priority, last use, row) order -- lowest priority first, least
// recently used within a priority -- until the pages taken reach `need`; a
// taken row is dropped (recomputed from its inputs later) when droppable and
// offloaded to host memory otherwise.  Returns the pages the taken rows hold.

enum TierAction { TIER_KEEP = 0, TIER_OFFLOAD = 1, TIER_DROP = 2 };

inline int64_t tier_plan(int n, const int32_t* priority, const int64_t* last_use, const int32_t* pages,
                         const int32_t* droppable, const int32_t* resident, const int32_t* pinned, int64_t need,
                         int32_t* action) {
  std::vector<int> order;
  for (int r = 0; r < n; ++r) {
    action[r] = TIER_KEEP;
    if (resident[r] && !pinned[r]) order.push_back(r);
  }
  if (need <= 0) return 0;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    if (priority[a] != priority[b]) return priority[a] < priority[b];
    if (last_use[a] != last_use[b]) return last_use[a] < last_use[b];
    return a < b;
  });
  int64_t freed = 0;
  for (int r : order) {
    if (freed >= need) break;
    action[r] = droppable[r] ? TIER_DROP : TIER_OFFLOAD;
    freed += pages[r];
  }
  return freed;
}

// ---------------------------------------------------------------------------
// pass planner: rows with pending tokens, packed in row order into passes of
// at most `pass_tokens` tokens (a row is never split: its count <= capacity
// <= pass_tokens).

struct Pass {
  int seg_begin, n_seg;  // into the call's segment arrays
  int tok_src;           // first token of the pass in the packed input
  int n_tok, max_len, max_end;
};

struct Plan {
  std::vector<int32_t> row, pos;  // per segment
  std::vector<int32_t> off;       // per pass: n_seg + 1 local offsets, passes back to back
  std::vector<Pass> passes;
};

// counts[b]: tokens to process for row b (0 = none); start[b]: first position.
inline Plan plan_passes(int batch, const int32_t* counts, const int32_t* start, int pass_tokens) {
  Plan p;
  int src = 0;
  Pass cur{0, 0, 0, 0, 0, 0};
  std::vector<int32_t> cur_off{0};
  auto flush = [&]() {
    if (cur.n_seg == 0) return;
    p.passes.push_back(cur);
    p.off.insert(p.off.end(), cur_off.begin(), cur_off.end());
    cur = Pass{(int)p.row.size(), 0, src, 0, 0, 0};
    cur_off.assign(1, 0);
  };
  cur.tok_src = 0;
  for (int b = 0; b < batch; ++b) {
    const int n = counts[b];
    if (n <= 0) continue;
    if (cur.n_tok + n > pass_tokens) flush();
    if (cur.n_seg == 0) { cur.seg_begin = (int)p.row.size(); cur.tok_src = src; }
    p.row.push_back(b);
    p.pos.push_back(start[b]);
    cur.n_seg++;
    cur.n_tok += n;
    cur.max_len = std::max(cur.max_len, n);
    cur.max_end = std::max(cur.max_end, start[b] + n);
    cur_off.push_back(cur.n_tok);
    src += n;
  }
  flush();
  return p;
}

// Each pass's segments by decreasing key count (pos + len; ties by index),
// as indices local to the pass, at the pass's first segment.
inline std::vector<int32_t> pass_orders(const Plan& p, const int32_t* counts) {
  std::vector<int32_t> ord(p.row.size());
  for (const Pass& ps : p.passes) {
    auto keys = [&](int i) { const int s = ps.seg_begin + i; return p.pos[s] + counts[p.row[s]]; };
    int32_t* o = ord.data() + ps.seg_begin;
    for (int i = 0; i < ps.n_seg; ++i) o[i] = i;
    std::stable_sort(o, o + ps.n_seg, [&](int a, int b) { return keys(a) > keys(b); });
  }
  return ord;
}

// Key splits of the decode attention.  One workgroup per (row, head) covers
// the row's keys in rounds of up to 8 waves x one key block; a split costs a
// second (merge) kernel of a few microseconds, which only pays when there are
// few (row, head) pairs and each would need many rounds: fewer than 128 pairs
// and a capacity above 2048 positions split into parts of at least 1024, for
// about 256 workgroups in all.
inline int decode_splits(int batch, int n_heads, int capacity) {
  const int pairs = batch * n_heads;
  if (pairs >= 128 || capacity <= 2048) return 1;
  const int s = (256 + pairs - 1) / pairs;
  return std::max(1, std::min(s, capacity / 1024));
}

}  // namespace ams
