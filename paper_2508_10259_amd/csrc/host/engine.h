// Engine: owns the host handles of a model and of a context and enqueues the
// forward passes.  All checks happen in the C ABI layer before these run.
#pragma once

#include <hip/hip_runtime.h>

#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "kernels.h"
#include "state.h"

namespace ams {

struct ams_weights_view {
  const void *w_q, *w_k, *w_v, *w_o, *w_gate, *w_up, *w_down;
  const float *g_attn, *g_ffn, *g_final;
  const void *embed, *head_bins;
};

struct Model {
  Cfg cfg;
  ModelLayout lay;
  int st = 0;  // storage type of the caller's arrays (kernels.h DType)
  int ct = 0;  // compute type of the packed weights, activations and K/V
  int device = 0;
  char* ws = nullptr;
  const void* embed = nullptr;  // caller's full table (referenced)
  int live_ctx = 0;

  const void* wqkv(int l) const { return ws + lay.wqkv + l * lay.per_layer_qkv; }
  const void* wo(int l) const { return ws + lay.wo + l * lay.per_layer_o; }
  const void* wgu(int l) const { return ws + lay.wgu + l * lay.per_layer_gu; }
  const void* wd(int l) const { return ws + lay.wd + l * lay.per_layer_d; }
  const void* head_bins() const { return ws + lay.head_bins; }
  const void* bin_embed() const { return ws + lay.bin_embed; }
  // the fragment-ordered copies (fp16 compute)
  const void* fqkv(int l) const { return ws + lay.fqkv + l * lay.per_layer_qkv; }
  const void* fo(int l) const { return ws + lay.fo + l * lay.per_layer_o; }
  const void* fgu(int l) const { return ws + lay.fgu + l * lay.per_layer_gu; }
  const void* fd(int l) const { return ws + lay.fd + l * lay.per_layer_d; }
  const void* fhead() const { return ws + lay.fhead; }
};

struct GraphKey {
  int n_actions;
  void* tokens;
  void* logits;
  const void* forced;
  bool operator<(const GraphKey& o) const {
    return std::tie(n_actions, tokens, logits, forced) < std::tie(o.n_actions, o.tokens, o.logits, o.forced);
  }
};

struct Ctx {
  Model* model = nullptr;
  CtxLayout lay;
  RowBook book;
  char* ws = nullptr;
  int splits = 1;
  int fused_grid = 0;  // workgroups of the persistent decode, 0 when it does not apply
  int split_o = 1, split_d = 1, split_a = 1;
  hipStream_t capture_stream = nullptr;
  // pinned host word the persistent decode sets when a barrier wait gives up
  // (host view, device view); read by the next call on the context
  volatile unsigned* status_host = nullptr;
  unsigned* status_dev = nullptr;
  std::map<GraphKey, hipGraphExec_t> graphs;
  std::vector<GraphKey> graph_lru;
  std::vector<int32_t> meta_host;  // staging of one call's pass metadata (kept until the next call)
  std::vector<int32_t> pt_host;      // the page table (-1: no page)
  std::vector<int32_t> pt_dev_host;  // staging of its last upload
  // pooled pages (created with a page count or prefix sharing): rows take pages
  // from `pool` when built and return them when invalidated; otherwise row b
  // keeps pages b * ppr .. b * ppr + ppr - 1 for the context's life
  bool pooled = false;
  PagePool pool;
  std::vector<uint64_t> keys_host;
  std::vector<int64_t> hk_rows_host;
  std::vector<XferRow> xfer_host;  // staging of the last host-tier call's descriptors

  // K/V page pools of layer l; row b's position t sits in page pt()[b * ppr + t / 64]
  void* kslab(int l) const { return ws + lay.kv + (size_t)(2 * l) * lay.slab_layer; }
  void* vslab(int l) const { return ws + lay.kv + (size_t)(2 * l + 1) * lay.slab_layer; }
  float* h() const { return (float*)(ws + lay.h); }
  void* u() const { return ws + lay.u; }
  float* qkv() const { return (float*)(ws + lay.qkv); }
  void* o() const { return ws + lay.o; }
  void* a() const { return ws + lay.a; }
  float* h_last() const { return (float*)(ws + lay.h_last); }
  void* h_last16() const { return ws + lay.h_last16; }
  void* h_last16lo() const { return ws + lay.h_last16lo; }
  void* hlo() const { return ws + lay.hlo; }
  void* olo() const { return ws + lay.olo; }
  void* alo() const { return ws + lay.alo; }
  float* kpart() const { return (float*)(ws + lay.kpart); }
  unsigned* wcnt() const { return (unsigned*)(ws + lay.wcnt); }
  float* part() const { return (float*)(ws + lay.part); }
  float* logits() const { return (float*)(ws + lay.logits); }
  float2* rope() const { return (float2*)(ws + lay.rope); }
  int32_t* lens() const { return (int32_t*)(ws + lay.lens); }
  int32_t* meta() const { return (int32_t*)(ws + lay.meta); }
  int32_t* pt() const { return (int32_t*)(ws + lay.pt); }
  KvPages pages() const { return KvPages{pt(), lay.ppr}; }
};

// Enqueue-level operations; each returns hipSuccess or the first failure and
// fills `err`.
hipError_t model_pack(Model& m, const ams_weights_view& w, hipStream_t s, std::string& err);
hipError_t ctx_init(Ctx& c, std::string& err);
// Runs every layer over counts[b] tokens of each row b at positions start[b]..;
// the tokens come from x packed row after row in row order, or, with src, from
// input tokens src[b].. of x.  Lengths afterwards: lens[b] += counts[b], or, with
// set_lens, lens[b] = lens_set[b] (counts[b] when lens_set is NULL) for the rows
// with counts[b] > 0.
hipError_t ctx_forward_tokens(Ctx& c, const void* x, const int32_t* counts, const int32_t* start, int set_lens,
                              hipStream_t s, std::string& err, const int32_t* src = nullptr,
                              const int32_t* lens_set = nullptr);
hipError_t ctx_decode(Ctx& c, int n_actions, int32_t* out_tokens, float* out_logits, const int32_t* forced,
                      hipStream_t s, std::string& err);
void ctx_release(Ctx& c);
// Builds the listed rows (strictly increasing; lens[i] tokens each, packed in
// order in `prefix`): pages first (the pool's shared prefix pages when the
// context shares them -- their keys hashed on the device and read back, the
// only synchronisation), then the forward passes over each row's tokens from
// its first unshared page on.  S_OK, S_ECAPACITY (no free page; nothing
// changed) or S_EHIP.
int ctx_build_rows(Ctx& c, const void* prefix, const int32_t* rows, int n_rows, const int32_t* lens, hipStream_t s,
                   std::string& err);
// Returns the listed rows' pages to the pool (pooled contexts; host only).
void ctx_release_rows(Ctx& c, const int32_t* rows, int n_rows);

// Host tier: copies the listed rows (lens[i] positions each) to / from the host
// images at host_dev[i] (device addresses of pinned host memory).  Reloading
// into a pooled context first takes fresh pages for the rows (S_ECAPACITY when
// there are not enough; nothing changed) and sets their device lengths.
int ctx_offload_rows(Ctx& c, const int32_t* rows, int n_rows, const int32_t* lens, void* const* host_dev,
                     hipStream_t s, std::string& err);
int ctx_reload_rows(Ctx& c, const int32_t* rows, int n_rows, const int32_t* lens, void* const* host_dev,
                    hipStream_t s, std::string& err);

// Flow-matching sampling of every row's action chunk (x: device fp32
// [batch][n_tokens][a], updated in place): n_steps Euler steps from tau0, each
// running the chunk's tokens through every layer at positions lens[b].. (their
// K/V are scratch) between the head's input and output projections.
struct FlowHeadView {
  const void *w_in, *w_t, *w_out;
  int a, n_tokens;
};
hipError_t ctx_flow(Ctx& c, const FlowHeadView& fh, float* x, float tau0, int n_steps, hipStream_t s,
                    std::string& err);

// Takes in an error a kernel of an earlier call reported asynchronously (see
// RowBook::absorb_async_error) and clears the word.
int ctx_absorb_status(Ctx& c, std::string& err);

}  // namespace ams
