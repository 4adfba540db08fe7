// C ABI (include/ams.h): argument, state and capacity checks, device-pointer
// range checks, then the engine.  Nothing is enqueued before every check has
// passed; a HIP failure after that invalidates the context.
#include "ams.h"

#include <string.h>

#include <algorithm>

#include <string>
#include <vector>

#include "engine.h"
#include "kernels.h"

struct ams_model {
  ams::Model m;
};
struct ams_ctx {
  ams::Ctx c;
};

namespace {

thread_local std::string g_err;

ams_status fail(int s, const std::string& msg) {
  g_err = msg;
  return (ams_status)s;
}

ams::Cfg to_cfg(const ams_model_cfg& c) {
  return ams::Cfg{c.n_layers, c.d_model, c.n_heads, c.head_dim, c.d_ffn, c.vocab, c.n_bins,
                  c.rms_eps, c.rope_theta, c.dtype};
}

bool is_gfx950(int dev) {
  hipDeviceProp_t p;
  if (hipGetDeviceProperties(&p, dev) != hipSuccess) return false;
  return strncmp(p.gcnArchName, "gfx950", 6) == 0;
}

// Current device must be a gfx950.
int current_device(int* dev, std::string& err) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
    err = "no HIP device";
    return ams::S_ENODEV;
  }
  if (hipGetDevice(dev) != hipSuccess) {
    err = "hipGetDevice failed";
    return ams::S_ENODEV;
  }
  if (!is_gfx950(*dev)) {
    err = "current device is not a gfx950";
    return ams::S_ENODEV;
  }
  return ams::S_OK;
}

// [p, p + bytes) must lie inside one device allocation of `dev`.
bool dev_range(const void* p, size_t bytes, int dev, const char* what, std::string& err) {
  if (!p) {
    err = std::string(what) + " is NULL";
    return false;
  }
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess || a.type != hipMemoryTypeDevice || a.device != dev) {
    (void)hipGetLastError();
    err = std::string(what) + " is not device memory of the current device";
    return false;
  }
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) != hipSuccess) {
    (void)hipGetLastError();
    err = std::string(what) + ": allocation range unknown";
    return false;
  }
  if ((const char*)p + bytes > (const char*)base + size) {
    err = std::string(what) + " is smaller than " + std::to_string(bytes) + " bytes";
    return false;
  }
  return true;
}

bool aligned256(const void* p) { return ((uintptr_t)p & 255) == 0; }

}  // namespace

extern "C" {

const char* ams_status_str(int32_t s) {
  switch (s) {
    case AMS_OK: return "AMS_OK";
    case AMS_EINVAL: return "AMS_EINVAL";
    case AMS_ESTATE: return "AMS_ESTATE";
    case AMS_ECAPACITY: return "AMS_ECAPACITY";
    case AMS_ENODEV: return "AMS_ENODEV";
    case AMS_EHIP: return "AMS_EHIP";
    case AMS_ENOMEM: return "AMS_ENOMEM";
    default: return "AMS_UNKNOWN";
  }
}

const char* ams_last_error(void) { return g_err.c_str(); }

int32_t ams_device_count(void) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  int k = 0;
  for (int i = 0; i < n; ++i) k += is_gfx950(i);
  return k;
}

size_t ams_model_workspace_bytes(const ams_model_cfg* cfg) {
  if (!cfg) return 0;
  std::string e;
  const ams::Cfg c = to_cfg(*cfg);
  if (ams::check_cfg(c, e) != ams::S_OK) return 0;
  return ams::model_layout(c).total;
}

ams_status ams_model_create(const ams_model_cfg* cfg, const ams_weights* w, void* ws, size_t ws_bytes, void* stream,
                            ams_model** out) {
  g_err.clear();
  if (!cfg || !w || !out) return fail(AMS_EINVAL, "cfg, weights and out must not be NULL");
  const ams::Cfg c = to_cfg(*cfg);
  std::string e;
  if (int s = ams::check_cfg(c, e)) return fail(s, e);
  const ams::ModelLayout lay = ams::model_layout(c);
  if (!ws) return fail(AMS_EINVAL, "workspace is NULL");
  if (!aligned256(ws)) return fail(AMS_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < lay.total) return fail(AMS_ENOMEM, "model workspace too small: need " + std::to_string(lay.total));
  const void* ptrs[] = {w->w_q, w->w_k, w->w_v, w->w_o, w->w_gate, w->w_up, w->w_down,
                        w->g_attn, w->g_ffn, w->g_final, w->embed, w->head_bins};
  for (const void* p : ptrs)
    if (!p) return fail(AMS_EINVAL, "a weight pointer is NULL");
  int dev = 0;
  if (int s = current_device(&dev, e)) return fail(s, e);
  const size_t es = ams::elem_size(c), d = c.d_model, F = c.d_ffn, L = c.n_layers;
  struct {
    const void* p;
    size_t bytes;
    const char* what;
  } chk[] = {
      {w->w_q, L * d * d * es, "w_q"},         {w->w_k, L * d * d * es, "w_k"},
      {w->w_v, L * d * d * es, "w_v"},         {w->w_o, L * d * d * es, "w_o"},
      {w->w_gate, L * F * d * es, "w_gate"},   {w->w_up, L * F * d * es, "w_up"},
      {w->w_down, L * d * F * es, "w_down"},   {w->g_attn, L * d * 4, "g_attn"},
      {w->g_ffn, L * d * 4, "g_ffn"},          {w->g_final, d * 4, "g_final"},
      {w->embed, (size_t)c.vocab * d * es, "embed"}, {w->head_bins, (size_t)c.n_bins * d * es, "head_bins"},
      {ws, lay.total, "model workspace"},
  };
  for (auto& k : chk)
    if (!dev_range(k.p, k.bytes, dev, k.what, e)) return fail(AMS_EINVAL, e);

  ams_model* m = new ams_model();
  m->m.cfg = c;
  m->m.lay = lay;
  m->m.device = dev;
  m->m.ws = (char*)ws;
  m->m.embed = w->embed;
  m->m.st = c.dtype == AMS_F32 ? ams::DT_F32 : ams::DT_BF16;
  m->m.ct = c.dtype == AMS_F32 ? ams::DT_F32 : ams::DT_F16;
  const ams::ams_weights_view v{w->w_q,    w->w_k,  w->w_v,    w->w_o,     w->w_gate, w->w_up,
                                w->w_down, w->g_attn, w->g_ffn, w->g_final, w->embed,  w->head_bins};
  if (ams::model_pack(m->m, v, (hipStream_t)stream, e) != hipSuccess) {
    delete m;
    return fail(AMS_EHIP, e);
  }
  *out = m;
  return AMS_OK;
}

void ams_model_destroy(ams_model* m) { delete m; }

ams_status ams_embed_ids(const ams_model* m, const int32_t* ids, int32_t n, void* out, void* stream) {
  g_err.clear();
  if (!m) return fail(AMS_EINVAL, "model is NULL");
  if (n < 0) return fail(AMS_EINVAL, "n must be >= 0");
  if (n == 0) return AMS_OK;
  const ams::Cfg& c = m->m.cfg;
  std::string e;
  if (!dev_range(ids, (size_t)n * 4, m->m.device, "ids", e)) return fail(AMS_EINVAL, e);
  if (!dev_range(out, (size_t)n * c.d_model * ams::elem_size(c), m->m.device, "out", e)) return fail(AMS_EINVAL, e);
  hipError_t r = ams::embed_rows(m->m.st, m->m.embed, ids, n, c.d_model, c.vocab, out, (hipStream_t)stream);
  if (r != hipSuccess) return fail(AMS_EHIP, std::string("embed: ") + hipGetErrorString(r));
  return AMS_OK;
}

size_t ams_ctx_workspace_bytes(const ams_model_cfg* cfg, int32_t batch, int32_t capacity, int32_t max_pass_tokens) {
  if (!cfg) return 0;
  std::string e;
  const ams::Cfg c = to_cfg(*cfg);
  if (ams::check_cfg(c, e) != ams::S_OK) return 0;
  if (ams::check_ctx_args(c, batch, capacity, max_pass_tokens, e) != ams::S_OK) return 0;
  return ams::ctx_layout(c, batch, capacity, max_pass_tokens).total;
}

static int check_paged(int batch, int capacity, int32_t n_pages, int32_t flags, std::string& e) {
  if (flags & ~AMS_CTX_SHARE_PREFIX) {
    e = "unknown context flags";
    return AMS_EINVAL;
  }
  if (n_pages < 0 || (int64_t)n_pages > (int64_t)batch * (capacity / 64)) {
    e = "n_pages must be in [0, batch * capacity / 64]";
    return AMS_EINVAL;
  }
  return AMS_OK;
}

size_t ams_ctx_workspace_bytes_paged(const ams_model_cfg* cfg, int32_t batch, int32_t capacity,
                                     int32_t max_pass_tokens, int32_t n_pages, int32_t flags) {
  if (!cfg) return 0;
  std::string e;
  const ams::Cfg c = to_cfg(*cfg);
  if (ams::check_cfg(c, e) != ams::S_OK) return 0;
  if (ams::check_ctx_args(c, batch, capacity, max_pass_tokens, e) != ams::S_OK) return 0;
  if (check_paged(batch, capacity, n_pages, flags, e) != AMS_OK) return 0;
  return ams::ctx_layout(c, batch, capacity, max_pass_tokens, n_pages, flags & AMS_CTX_SHARE_PREFIX).total;
}

static ams_status ctx_create(ams_model* m, int32_t batch, int32_t capacity, int32_t max_pass_tokens,
                             int32_t n_pages, int32_t flags, bool pooled, void* ws, size_t ws_bytes, ams_ctx** out) {
  g_err.clear();
  if (!m || !out) return fail(AMS_EINVAL, "model and out must not be NULL");
  std::string e;
  if (int s = ams::check_ctx_args(m->m.cfg, batch, capacity, max_pass_tokens, e)) return fail(s, e);
  if (int s = check_paged(batch, capacity, n_pages, flags, e)) return fail(s, e);
  const ams::CtxLayout lay =
      ams::ctx_layout(m->m.cfg, batch, capacity, max_pass_tokens, n_pages, flags & AMS_CTX_SHARE_PREFIX);
  if (!ws) return fail(AMS_EINVAL, "workspace is NULL");
  if (!aligned256(ws)) return fail(AMS_EINVAL, "workspace must be 256-byte aligned");
  if (ws_bytes < lay.total) return fail(AMS_ENOMEM, "context workspace too small: need " + std::to_string(lay.total));
  if (!dev_range(ws, lay.total, m->m.device, "context workspace", e)) return fail(AMS_EINVAL, e);
  ams_ctx* c = new ams_ctx();
  c->c.model = &m->m;
  c->c.lay = lay;
  c->c.ws = (char*)ws;
  c->c.pooled = pooled;
  c->c.book.init(batch, capacity);
  if (ams::ctx_init(c->c, e) != hipSuccess) {
    ams::ctx_release(c->c);
    delete c;
    return fail(AMS_EHIP, e);
  }
  m->m.live_ctx++;
  *out = c;
  return AMS_OK;
}

ams_status ams_ctx_create(ams_model* m, int32_t batch, int32_t capacity, int32_t max_pass_tokens, void* ws,
                          size_t ws_bytes, ams_ctx** out) {
  return ctx_create(m, batch, capacity, max_pass_tokens, 0, 0, false, ws, ws_bytes, out);
}

ams_status ams_ctx_create_paged(ams_model* m, int32_t batch, int32_t capacity, int32_t max_pass_tokens,
                                int32_t n_pages, int32_t flags, void* ws, size_t ws_bytes, ams_ctx** out) {
  return ctx_create(m, batch, capacity, max_pass_tokens, n_pages, flags, true, ws, ws_bytes, out);
}

ams_status ams_ctx_pages(const ams_ctx* c, int32_t* page_table, int32_t* refs, int32_t* pages_in_use) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  const ams::Ctx& x = c->c;
  if (page_table) std::copy(x.pt_host.begin(), x.pt_host.end(), page_table);
  if (refs) {
    if (x.pooled) std::copy(x.pool.refs.begin(), x.pool.refs.end(), refs);
    else
      for (int p = 0; p < x.lay.n_pages; ++p) refs[p] = 1;
  }
  if (pages_in_use) *pages_in_use = x.pooled ? x.pool.in_use() : x.lay.n_pages;
  return AMS_OK;
}

void ams_ctx_destroy(ams_ctx* c) {
  if (!c) return;
  ams::ctx_release(c->c);
  c->c.model->live_ctx--;
  delete c;
}

ams_status ams_ctx_build(ams_ctx* c, const void* prefix, const int32_t* lens, void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  // a rebuild replaces whatever an earlier failed decode left behind
  (void)ams::ctx_absorb_status(x, e);
  e.clear();
  if (int s = x.book.check_build(lens, e)) return fail(s, e);
  size_t tot = 0;
  for (int b = 0; b < x.lay.batch; ++b) tot += (size_t)lens[b];
  const ams::Cfg& m = x.model->cfg;
  if (!dev_range(prefix, tot * m.d_model * ams::elem_size(m), x.model->device, "prefix", e))
    return fail(AMS_EINVAL, e);
  if (x.lay.share && ((uintptr_t)prefix & 15) != 0) return fail(AMS_EINVAL, "prefix must be 16-byte aligned");
  std::vector<int32_t> rows(x.lay.batch);
  for (int b = 0; b < x.lay.batch; ++b) rows[b] = b;
  if (int s = ams::ctx_build_rows(x, prefix, rows.data(), x.lay.batch, lens, (hipStream_t)stream, e)) {
    if (s == AMS_EHIP) {
      x.book.invalidate();
      ams::ctx_release_rows(x, rows.data(), x.lay.batch);
    }
    return fail(s, e);
  }
  x.book.commit_build(lens);
  return AMS_OK;
}

ams_status ams_ctx_step(ams_ctx* c, const void* new_tokens, const int32_t* new_lens, int32_t n_actions,
                        int32_t* out_tokens, float* out_logits, const int32_t* forced, void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x, e)) return fail(s, e);
  if (int s = x.book.check_step(new_lens, n_actions, e)) return fail(s, e);
  const ams::Cfg& m = x.model->cfg;
  const int B = x.lay.batch, dev = x.model->device;
  const size_t BA = (size_t)B * n_actions;
  if (!dev_range(out_tokens, BA * 4, dev, "out_tokens", e)) return fail(AMS_EINVAL, e);
  if (out_logits && !dev_range(out_logits, BA * m.n_bins * 4, dev, "out_logits", e)) return fail(AMS_EINVAL, e);
  if (forced && !dev_range(forced, BA * 4, dev, "forced", e)) return fail(AMS_EINVAL, e);
  size_t n_new = 0;
  if (new_lens)
    for (int b = 0; b < B; ++b) n_new += (size_t)new_lens[b];
  if (n_new > 0 && !dev_range(new_tokens, n_new * m.d_model * ams::elem_size(m), dev, "new_tokens", e))
    return fail(AMS_EINVAL, e);

  hipStream_t s = (hipStream_t)stream;
  if (n_new > 0) {
    if (ams::ctx_forward_tokens(x, new_tokens, new_lens, x.book.len.data(), 0, s, e) != hipSuccess) {
      x.book.invalidate();
      return fail(AMS_EHIP, e);
    }
    x.book.commit_new(new_lens);
  }
  if (ams::ctx_decode(x, n_actions, out_tokens, out_logits, forced, s, e) != hipSuccess) {
    x.book.invalidate();
    return fail(AMS_EHIP, e);
  }
  return AMS_OK;
}

ams_status ams_ctx_build_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, const void* prefix,
                              const int32_t* lens, void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x, e)) return fail(s, e);
  if (int s = x.book.check_build_rows(rows, n_rows, lens, e)) return fail(s, e);
  size_t tot = 0;
  for (int i = 0; i < n_rows; ++i) tot += (size_t)lens[i];
  const ams::Cfg& m = x.model->cfg;
  if (!dev_range(prefix, tot * m.d_model * ams::elem_size(m), x.model->device, "prefix", e))
    return fail(AMS_EINVAL, e);
  if (x.lay.share && ((uintptr_t)prefix & 15) != 0) return fail(AMS_EINVAL, "prefix must be 16-byte aligned");
  if (int s = ams::ctx_build_rows(x, prefix, rows, n_rows, lens, (hipStream_t)stream, e)) {
    if (s == AMS_EHIP) {
      x.book.invalidate();
      std::vector<int32_t> all(x.lay.batch);
      for (int b = 0; b < x.lay.batch; ++b) all[b] = b;
      ams::ctx_release_rows(x, all.data(), x.lay.batch);
    }
    return fail(s, e);
  }
  x.book.commit_build_rows(rows, n_rows, lens);
  return AMS_OK;
}

ams_status ams_ctx_append(ams_ctx* c, const void* new_tokens, const int32_t* new_lens, void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x, e)) return fail(s, e);
  if (int s = x.book.check_append(new_lens, e)) return fail(s, e);
  const ams::Cfg& m = x.model->cfg;
  size_t n_new = 0;
  for (int b = 0; b < x.lay.batch; ++b) n_new += (size_t)new_lens[b];
  if (n_new == 0) return AMS_OK;
  if (!dev_range(new_tokens, n_new * m.d_model * ams::elem_size(m), x.model->device, "new_tokens", e))
    return fail(AMS_EINVAL, e);
  if (ams::ctx_forward_tokens(x, new_tokens, new_lens, x.book.len.data(), 0, (hipStream_t)stream, e) != hipSuccess) {
    x.book.invalidate();
    return fail(AMS_EHIP, e);
  }
  x.book.commit_new(new_lens);
  return AMS_OK;
}

ams_status ams_ctx_invalidate_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  std::string e;
  if (int s = c->c.book.check_rows(rows, n_rows, e)) return fail(s, e);
  c->c.book.invalidate_rows(rows, n_rows);
  ams::ctx_release_rows(c->c, rows, n_rows);
  return AMS_OK;
}

size_t ams_index_hash_workspace_bytes(size_t n_bytes, int32_t seg_bytes) {
  if (n_bytes == 0 || seg_bytes < 16 || seg_bytes > 65536 || seg_bytes % 16) return 0;
  return ((n_bytes + seg_bytes - 1) / seg_bytes) * 8;
}

ams_status ams_index_hash(const void* data, size_t n_bytes, int32_t seg_bytes, void* ws, size_t ws_bytes,
                          uint64_t* out_hash, void* stream) {
  g_err.clear();
  std::string e;
  if (n_bytes == 0) return fail(AMS_EINVAL, "n_bytes must be >= 1");
  if (seg_bytes < 16 || seg_bytes > 65536 || seg_bytes % 16)
    return fail(AMS_EINVAL, "seg_bytes must be a multiple of 16 in [16, 65536]");
  const uint64_t k = (n_bytes + seg_bytes - 1) / seg_bytes;
  if (k > 0x7FFFFFFFull) return fail(AMS_EINVAL, "too many segments (more than 2^31 - 1)");
  if (((uintptr_t)data & 15) != 0) return fail(AMS_EINVAL, "data must be 16-byte aligned");
  if (((uintptr_t)ws & 7) != 0 || ((uintptr_t)out_hash & 7) != 0)
    return fail(AMS_EINVAL, "ws and out_hash must be 8-byte aligned");
  if (ws_bytes < k * 8) return fail(AMS_ENOMEM, "index workspace too small: need " + std::to_string(k * 8));
  int dev = 0;
  if (int s = current_device(&dev, e)) return fail(s, e);
  if (!dev_range(data, n_bytes, dev, "data", e) || !dev_range(ws, k * 8, dev, "ws", e) ||
      !dev_range(out_hash, 8, dev, "out_hash", e))
    return fail(AMS_EINVAL, e);
  hipStream_t st = (hipStream_t)stream;
  hipError_t r = ams::hash_segments(data, n_bytes, seg_bytes, (uint64_t*)ws, st);
  if (r == hipSuccess) r = ams::hash_merge((const uint64_t*)ws, k, n_bytes, out_hash, st);
  if (r != hipSuccess) return fail(AMS_EHIP, std::string("index hash: ") + hipGetErrorString(r));
  return AMS_OK;
}

ams_status ams_index_hash_noalloc(const void* data, size_t n_bytes, int32_t seg_bytes, uint64_t* out_hash,
                                  void* stream) {
  g_err.clear();
  std::string e;
  if (n_bytes == 0) return fail(AMS_EINVAL, "n_bytes must be >= 1");
  if (seg_bytes < 16 || seg_bytes > 65536 || seg_bytes % 16)
    return fail(AMS_EINVAL, "seg_bytes must be a multiple of 16 in [16, 65536]");
  const uint64_t k = (n_bytes + seg_bytes - 1) / seg_bytes;
  if (k > ams::INDEX_NOALLOC_MAX_SEGMENTS)
    return fail(AMS_EINVAL, "ams_index_hash_noalloc: " + std::to_string(k) + " segments exceed its scratch of " +
                                std::to_string(ams::INDEX_NOALLOC_MAX_SEGMENTS) + " (use ams_index_hash)");
  if (((uintptr_t)data & 15) != 0) return fail(AMS_EINVAL, "data must be 16-byte aligned");
  if (((uintptr_t)out_hash & 7) != 0) return fail(AMS_EINVAL, "out_hash must be 8-byte aligned");
  int dev = 0;
  if (int s = current_device(&dev, e)) return fail(s, e);
  if (!dev_range(data, n_bytes, dev, "data", e) || !dev_range(out_hash, 8, dev, "out_hash", e))
    return fail(AMS_EINVAL, e);
  uint64_t* scratch = nullptr;
  hipError_t r = ams::index_noalloc_scratch(dev, &scratch);
  if (r != hipSuccess) return fail(AMS_EHIP, std::string("index scratch: ") + hipGetErrorString(r));
  hipStream_t st = (hipStream_t)stream;
  r = ams::hash_segments(data, n_bytes, seg_bytes, scratch, st);
  if (r == hipSuccess) r = ams::hash_merge(scratch, k, n_bytes, out_hash, st);
  if (r != hipSuccess) return fail(AMS_EHIP, std::string("index hash: ") + hipGetErrorString(r));
  return AMS_OK;
}

namespace {
constexpr uint32_t ROW_IMAGE_MAGIC = 0x52534D41u;  // "AMSR"
struct RowImageHeader {
  uint32_t magic, version;
  int32_t len, n_layers, d_model, head_dim, n_heads, dtype;
};

// Device address of pinned host memory (EINVAL when `p` is not pinned and mapped).
bool host_device_ptr(const void* p, void** dev, std::string& err) {
  hipPointerAttribute_t a;
  if (!p || hipPointerGetAttributes(&a, p) != hipSuccess || a.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    err = "a host buffer is not pinned host memory (hipHostMalloc)";
    return false;
  }
  if (hipHostGetDevicePointer(dev, (void*)p, 0) != hipSuccess) {
    (void)hipGetLastError();
    err = "a host buffer is not mapped for the device";
    return false;
  }
  return true;
}
}  // namespace

size_t ams_ctx_row_host_bytes(const ams_ctx* c, int32_t len) {
  if (!c || len < 1 || len > c->c.lay.capacity) return 0;
  return ams::row_host_bytes(c->c.model->cfg, len);
}

ams_status ams_ctx_offload_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, void* const* host, void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x, e)) return fail(s, e);
  if (int s = x.book.check_offload(rows, n_rows, e)) return fail(s, e);
  if (!host) return fail(AMS_EINVAL, "host is NULL");
  std::vector<void*> dev(n_rows);
  std::vector<int32_t> lens(n_rows);
  for (int i = 0; i < n_rows; ++i) {
    if (!host_device_ptr(host[i], &dev[i], e)) return fail(AMS_EINVAL, e);
    if (((uintptr_t)host[i] & 15) != 0) return fail(AMS_EINVAL, "host buffers must be 16-byte aligned");
    lens[i] = x.book.len[rows[i]];
  }
  const ams::Cfg& m = x.model->cfg;
  for (int i = 0; i < n_rows; ++i) {
    RowImageHeader hd{ROW_IMAGE_MAGIC, 1u, lens[i], m.n_layers, m.d_model, m.head_dim, m.n_heads, m.dtype};
    memcpy(host[i], &hd, sizeof(hd));
  }
  if (int s = ams::ctx_offload_rows(x, rows, n_rows, lens.data(), dev.data(), (hipStream_t)stream, e)) {
    x.book.invalidate();
    return fail(s, e);
  }
  x.book.offload_rows(rows, n_rows);
  return AMS_OK;
}

ams_status ams_ctx_reload_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, const void* const* host,
                               void* stream) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  ams::Ctx& x = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x, e)) return fail(s, e);
  if (int s = x.book.check_reload(rows, n_rows, e)) return fail(s, e);
  if (!host) return fail(AMS_EINVAL, "host is NULL");
  const ams::Cfg& m = x.model->cfg;
  std::vector<void*> dev(n_rows);
  std::vector<int32_t> lens(n_rows);
  for (int i = 0; i < n_rows; ++i) {
    if (!host_device_ptr(host[i], &dev[i], e)) return fail(AMS_EINVAL, e);
    if (((uintptr_t)host[i] & 15) != 0) return fail(AMS_EINVAL, "host buffers must be 16-byte aligned");
    RowImageHeader hd;
    memcpy(&hd, host[i], sizeof(hd));
    if (hd.magic != ROW_IMAGE_MAGIC || hd.version != 1u || hd.n_layers != m.n_layers || hd.d_model != m.d_model ||
        hd.head_dim != m.head_dim || hd.n_heads != m.n_heads || hd.dtype != m.dtype)
      return fail(AMS_EINVAL, "host buffer " + std::to_string(i) + " holds no row image of this model");
    if (hd.len < 1 || hd.len > x.lay.capacity)
      return fail(AMS_ECAPACITY, "host buffer " + std::to_string(i) + ": row longer than the capacity");
    lens[i] = hd.len;
  }
  if (int s = ams::ctx_reload_rows(x, rows, n_rows, lens.data(), dev.data(), (hipStream_t)stream, e)) {
    if (s == AMS_EHIP) x.book.invalidate();
    return fail(s, e);
  }
  x.book.commit_build_rows(rows, n_rows, lens.data());
  return AMS_OK;
}

ams_status ams_ctx_row_states(const ams_ctx* c, int32_t* states) {
  g_err.clear();
  if (!c || !states) return fail(AMS_EINVAL, "context and states must not be NULL");
  for (int b = 0; b < c->c.lay.batch; ++b) states[b] = c->c.book.row_state[b];
  return AMS_OK;
}

ams_status ams_ctx_flow(ams_ctx* c, const ams_flow_head* head, float* x, float tau0, int32_t n_steps,
                        void* stream) {
  g_err.clear();
  if (!c || !head) return fail(AMS_EINVAL, "context and head must not be NULL");
  ams::Ctx& x_ = c->c;
  std::string e;
  if (int s = ams::ctx_absorb_status(x_, e)) return fail(s, e);
  if (x_.book.state != ams::READY) return fail(AMS_ESTATE, "context (or a row of it) is not built");
  const int a = head->action_dim, T = head->n_tokens;
  if (a < 1 || a > ams::FLOW_MAX_ACTION_DIM) return fail(AMS_EINVAL, "action_dim must be in [1, 256]");
  if (T < 1) return fail(AMS_EINVAL, "n_tokens must be >= 1");
  if (n_steps < 0) return fail(AMS_EINVAL, "n_steps must be >= 0");
  if (!(tau0 >= 0.f && tau0 < 1.f)) return fail(AMS_EINVAL, "tau0 must be in [0, 1)");
  for (int b = 0; b < x_.lay.batch; ++b)
    if (x_.book.len[b] + T > x_.lay.capacity)
      return fail(AMS_ECAPACITY, "row " + std::to_string(b) + ": context + action tokens exceed the capacity");
  const ams::Cfg& m = x_.model->cfg;
  const size_t es = ams::elem_size(m), d = m.d_model, B = x_.lay.batch;
  const int dev = x_.model->device;
  if (!dev_range(head->w_in, d * a * es, dev, "w_in", e) || !dev_range(head->w_t, d * es, dev, "w_t", e) ||
      !dev_range(head->w_out, (size_t)a * d * es, dev, "w_out", e) ||
      !dev_range(x, B * (size_t)T * a * 4, dev, "x", e))
    return fail(AMS_EINVAL, e);
  const ams::FlowHeadView fh{head->w_in, head->w_t, head->w_out, a, T};
  if (ams::ctx_flow(x_, fh, x, tau0, n_steps, (hipStream_t)stream, e) != hipSuccess) {
    x_.book.invalidate();
    return fail(AMS_EHIP, e);
  }
  return AMS_OK;
}

ams_status ams_tier_plan(int32_t n_rows, const int32_t* priority, const int64_t* last_use, const int32_t* pages,
                         const int32_t* droppable, const int32_t* resident, const int32_t* pinned,
                         int64_t pages_needed, int32_t* action, int64_t* pages_freed) {
  g_err.clear();
  if (n_rows < 0) return fail(AMS_EINVAL, "n_rows must be >= 0");
  if (n_rows > 0 && (!priority || !last_use || !pages || !droppable || !resident || !pinned || !action))
    return fail(AMS_EINVAL, "an array is NULL");
  const int64_t f = ams::tier_plan(n_rows, priority, last_use, pages, droppable, resident, pinned, pages_needed,
                                   action);
  if (pages_freed) *pages_freed = f;
  return AMS_OK;
}

ams_status ams_ctx_invalidate(ams_ctx* c) {
  g_err.clear();
  if (!c) return fail(AMS_EINVAL, "context is NULL");
  c->c.book.invalidate();
  std::vector<int32_t> all(c->c.lay.batch);
  for (int b = 0; b < c->c.lay.batch; ++b) all[b] = b;
  ams::ctx_release_rows(c->c, all.data(), c->c.lay.batch);
  return AMS_OK;
}

ams_status ams_ctx_lengths(const ams_ctx* c, int32_t* lens) {
  g_err.clear();
  if (!c || !lens) return fail(AMS_EINVAL, "context and lens must not be NULL");
  for (int b = 0; b < c->c.lay.batch; ++b) lens[b] = c->c.book.len[b];
  return AMS_OK;
}

int32_t ams_ctx_state(const ams_ctx* c) {
  if (!c) return AMS_EINVAL;
  // an asynchronously reported decode failure makes the context INVALID
  if (c->c.status_host && *c->c.status_host) return ams::INVALID;
  return c->c.book.state;
}

int32_t ams_ctx_persistent_decode(const ams_ctx* c) {
  if (!c) return AMS_EINVAL;
  return c->c.fused_grid > 0 ? 1 : 0;
}

}  // extern "C"
