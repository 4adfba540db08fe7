/*
 * ams.h -- C ABI of the cached-context action decoder on one AMD MI355X (gfx950).
 *
 * What the library computes
 *   A decoder-only transformer (Llama-style: RMSNorm, rotary position
 *   embedding, causal multi-head attention, SwiGLU feed-forward) that emits
 *   discretised action tokens greedily over the last n_bins vocabulary ids.
 *   The step-invariant prefix of each episode (instruction tokens and
 *   unchanged observation tokens) stays resident in device memory as a
 *   per-layer key/value cache -- the "action context" of the paper (section
 *   3.2.1, Constructing the Action Context): cached intermediate state is
 *   reused by the next inference so only new tokens are computed, and the
 *   new tokens' K/V are added after the inference.  Discarding a context and
 *   re-inferring from fresh environment data follows the common part of the
 *   paper's exception handler (section 3.3, Handler).  Control logic stays on
 *   the host; every arithmetic step runs in the library's HIP kernels
 *   (section 4 places control on the CPU and context on the GPU).
 *
 * Conventions
 *   - Device pointers come from the caller (e.g. torch tensors' data_ptr());
 *     `stream` is a hipStream_t (NULL = the legacy default stream).
 *   - The caller owns every device buffer: weights, workspaces, inputs and
 *     outputs.  They must outlive the handles that use them.  The library
 *     allocates no device memory; it owns host-side handles, metadata,
 *     captured HIP graphs and one pinned host word per context through which
 *     a kernel reports a failure to the next call.
 *   - Calls are asynchronous: they return after enqueueing on `stream`;
 *     outputs are valid once the caller synchronises that stream.
 *   - Every argument, state and capacity check happens before anything is
 *     enqueued.  A call that fails a check returns a negative status and
 *     changes nothing.  A failed HIP enqueue returns AMS_EHIP and moves the
 *     context to the INVALID state.  ams_last_error() gives a message
 *     (thread-local, valid until the next call on the same thread).
 *   - A model is read-only after creation and may be shared by contexts.
 *     A context must be used by one host thread and one stream at a time.
 *
 * Data types and layouts (row-major throughout)
 *   dtype AMS_F32: weights, embeddings and K/V in fp32; all arithmetic fp32.
 *   dtype AMS_BF16: the caller's weights and embeddings are bf16.  The packed
 *     weights, GEMM inputs (activations) and the K/V cache are fp16 (same
 *     bytes and MFMA rate as bf16, three more mantissa bits); bf16 weights
 *     convert exactly unless |w| < 2^-14, where the fp16 subnormal is within
 *     2^-25.  fp16 values saturate at +-65504.  Accumulation, residual
 *     stream, norm statistics, softmax and logits are fp32.
 *   A weight matrix maps an input vector x to W x and is stored [out][in].
 *
 * Context state machine (each row has its own state; the context is READY
 * when every row is, EMPTY while no row has been built, INVALID otherwise)
 *   create -> EMPTY;  build: EMPTY|READY|INVALID -> READY;
 *   step, append: READY -> READY (EMPTY or INVALID: AMS_ESTATE);
 *   invalidate: any -> INVALID;  invalidate_rows: the listed rows -> INVALID;
 *   build_rows: the listed rows -> READY.
 */
#ifndef AMS_H
#define AMS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ams_model ams_model;
typedef struct ams_ctx ams_ctx;

typedef enum {
  AMS_OK = 0,
  AMS_EINVAL = -1,    /* bad argument (NULL, out of range, inconsistent sizes) */
  AMS_ESTATE = -2,    /* context is not in a state that allows the call */
  AMS_ECAPACITY = -3, /* a row would exceed the context's token capacity */
  AMS_ENODEV = -4,    /* no usable gfx950 device */
  AMS_EHIP = -5,      /* a HIP runtime call failed */
  AMS_ENOMEM = -6     /* a workspace is smaller than required */
} ams_status;

typedef enum { AMS_F32 = 0, AMS_BF16 = 1 } ams_dtype;

/* Decoder dimensions.  d_model = n_heads * head_dim; head_dim even and at
 * most 128; d_model a multiple of 128; d_ffn a multiple of 128;
 * 0 < n_bins <= vocab, n_bins <= 1024.  rms_eps > 0, rope_theta > 1. */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, n_bins;
  float rms_eps;    /* RMSNorm: x / sqrt(mean(x^2) + rms_eps) * gain */
  float rope_theta; /* RoPE base: pair (i, i + head_dim/2) turns by t * theta^(-2i/head_dim) */
  int32_t dtype;    /* ams_dtype */
} ams_model_cfg;

/* Device pointers to the model's parameters (dtype = cfg.dtype unless fp32 is stated).
 * ams_model_create packs them into the model workspace -- each RMSNorm gain is
 * folded into the columns of the matrices that read the normalised vector
 * (W diag(g)) -- except `embed`, which ams_embed_ids reads and must outlive the
 * model. */
typedef struct {
  const void *w_q, *w_k, *w_v, *w_o; /* [n_layers][d][d] */
  const void *w_gate, *w_up;         /* [n_layers][d_ffn][d] */
  const void *w_down;                /* [n_layers][d][d_ffn] */
  const float *g_attn, *g_ffn;       /* [n_layers][d] fp32 RMSNorm gains */
  const float *g_final;              /* [d] fp32 final RMSNorm gain */
  const void *embed;                 /* [vocab][d] input embedding table */
  const void *head_bins;             /* [n_bins][d]: rows vocab-n_bins..vocab-1 of the output head */
} ams_weights;

/* ---- library ---------------------------------------------------------- */

/* Status name ("AMS_OK", ...); never NULL. */
const char* ams_status_str(int32_t status);
/* Message of the last failing call on this thread ("" if none); never NULL. */
const char* ams_last_error(void);
/* Number of visible gfx950 devices (0 when none or no HIP runtime). */
int32_t ams_device_count(void);

/* ---- model ------------------------------------------------------------ */

/* Bytes of device workspace ams_model_create needs for `cfg` (0 if cfg is invalid).
 * fp16 compute (bf16 and fp16 models) keeps each layer matrix and the action
 * head twice: row-major for the prefix passes and the decode of up to 8 rows
 * outside the persistent kernel, and in MFMA fragment order for the wider
 * decode passes and the persistent decode, so such a model needs about twice
 * its weight bytes. */
size_t ams_model_workspace_bytes(const ams_model_cfg* cfg);

/* Validates cfg and weights, then packs the weights into `ws` (device memory of
 * at least ams_model_workspace_bytes(cfg) bytes, 256-byte aligned) with
 * copies enqueued on `stream`.  The source weights may be freed once the
 * stream has passed the copies; `ws` and `embed` must outlive the model.
 * On success *out receives the handle.  Errors: AMS_EINVAL, AMS_ENOMEM,
 * AMS_ENODEV, AMS_EHIP. */
ams_status ams_model_create(const ams_model_cfg* cfg, const ams_weights* w, void* ws,
                            size_t ws_bytes, void* stream, ams_model** out);
void ams_model_destroy(ams_model* m); /* NULL is a no-op; destroy contexts first */

/* ---- text embedding --------------------------------------------------- */

/* out[i][:] = embed[ids[i]][:] for i < n (ids and out on the device, out of
 * shape [n][d] in the model dtype).  Ids outside [0, vocab) are clamped into
 * range by the kernel.  Prefix ingest for instruction tokens.
 * Errors: AMS_EINVAL, AMS_EHIP. */
ams_status ams_embed_ids(const ams_model* m, const int32_t* ids, int32_t n, void* out,
                         void* stream);

/* ---- action index ----------------------------------------------------- */

/* Paper section 3.2.3 (Action Compression, Virtual Action; Algorithm 1,
 * Two-Phase Hashing for Action Index): an input serialised to bytes is cut
 * into ceil(n_bytes / seg_bytes) segments of seg_bytes bytes (the last may be
 * shorter); phase 1 hashes every segment independently, phase 2 merges the
 * segment hashes in order into the index value.  The paper says only that
 * both hash functions are modular; here they are polynomial hashes modulo
 * p = 2^31 - 1 evaluated with two fixed bases each, the two 31-bit results
 * packed into one uint64 (first base in the low 32 bits):
 *   HashFunc1(B_i) = (sum_j u_j r^(seg_bytes/2 - 1 - j)) r + |B_i| mod p,
 *     u_j the 16-bit little-endian units of B_i zero-padded to seg_bytes,
 *     |B_i| its unpadded length; r = 0x2545F491, then 0x1B873593;
 *   H = HashFunc2(h_1..h_k) = (sum_i h_i q^(k - i)) q + n_bytes mod p,
 *     q = 0x3C6EF372, then 0x0A54FF53.
 * Bytes of workspace ams_index_hash needs: 8 per segment (0 if the sizes are
 * invalid). */
size_t ams_index_hash_workspace_bytes(size_t n_bytes, int32_t seg_bytes);

/* Two-phase hash of n_bytes >= 1 bytes of device memory `data` (16-byte
 * aligned); seg_bytes a multiple of 16 in [16, 65536].  `ws` (device, 8-byte
 * aligned, at least ams_index_hash_workspace_bytes bytes, caller-owned) holds
 * the phase-1 segment hashes h_1..h_k (uint64 each) when the call completes;
 * *out_hash (device uint64) receives H.  Asynchronous on `stream`.
 * Errors: AMS_EINVAL (sizes, alignment, pointers not on the current device),
 * AMS_ENOMEM (ws too small), AMS_ENODEV, AMS_EHIP. */
ams_status ams_index_hash(const void* data, size_t n_bytes, int32_t seg_bytes, void* ws, size_t ws_bytes,
                          uint64_t* out_hash, void* stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: the same
 * two-phase hash as ams_index_hash with no workspace argument.  The phase-1
 * segment hashes go to a static scratch array of the library (1 MiB, one copy
 * per device, held until the process ends), so at most 131072 segments
 * (n_bytes <= 131072 * seg_bytes) are accepted, else AMS_EINVAL.  The call
 * allocates nothing.  Calls on one device share the scratch: calls that
 * overlap (other streams, other host threads) race; calls on one stream are
 * ordered.  Other arguments and errors as ams_index_hash. */
ams_status ams_index_hash_noalloc(const void* data, size_t n_bytes, int32_t seg_bytes, uint64_t* out_hash,
                                  void* stream);

/* ---- context ---------------------------------------------------------- */

/* Bytes of device workspace a context needs: the K/V slab for `batch` rows of
 * `capacity` tokens (head-major [layer][K|V][row][head][capacity][head_dim])
 * plus activations for `max_pass_tokens` tokens per forward pass
 * (0 selects min(batch * capacity, 32768)).  0 if an argument is invalid. */
size_t ams_ctx_workspace_bytes(const ams_model_cfg* cfg, int32_t batch, int32_t capacity,
                               int32_t max_pass_tokens);

/* Creates a context of `batch` rows, each holding up to `capacity` tokens
 * (1 <= batch <= 1024, capacity a multiple of 64, capacity >= 64).  `ws` is
 * device memory of at least ams_ctx_workspace_bytes(...) bytes, 256-byte
 * aligned, owned by the caller.  State EMPTY.  Errors: AMS_EINVAL,
 * AMS_ENOMEM, AMS_EHIP. */
ams_status ams_ctx_create(ams_model* m, int32_t batch, int32_t capacity, int32_t max_pass_tokens,
                          void* ws, size_t ws_bytes, ams_ctx** out);
void ams_ctx_destroy(ams_ctx* c); /* NULL is a no-op */

/* Paper section 3.2.3 (Action Compression, Virtual Action): a context whose
 * K/V live in a pool of pages, each page holding 64 consecutive positions of
 * one row for every layer and head, with a reference count per page.  With
 * AMS_CTX_SHARE_PREFIX, building a row computes the page keys of its prefix --
 * the two-phase hash (ams_index_hash's functions, seg_bytes the largest power of
 * two <= 4096 dividing d_model * element size) of the row's prefix bytes up to
 * the end of each full page that does not hold its last token -- and every such
 * page whose key is already published (by another row, in this call or an
 * earlier one) is referenced instead of being computed and stored again; the
 * row computes its K/V from its first unshared page on.  Pages the row computes
 * are published under their keys.  Invalidating a row drops one reference to
 * each of its pages; a page whose count reaches zero returns to the pool and
 * leaves the index.  A build first reads the keys back from the device (it
 * synchronises `stream`).  Rows hold pages for their whole capacity from the
 * build on, so a pool smaller than batch * capacity / 64 pages fits the batch
 * when rows share enough prefix pages; a build that needs more pages than are
 * free fails with AMS_ECAPACITY and changes nothing.  Results equal an unshared
 * context's up to rounding (shared pages may come from a pass of other rows). */
#define AMS_CTX_SHARE_PREFIX 1

/* Bytes of workspace of a paged context: as ams_ctx_workspace_bytes with
 * n_pages K/V pages per layer pool (0: batch * capacity / 64) and `flags`
 * (0 or AMS_CTX_SHARE_PREFIX).  0 if an argument is invalid. */
size_t ams_ctx_workspace_bytes_paged(const ams_model_cfg* cfg, int32_t batch, int32_t capacity,
                                     int32_t max_pass_tokens, int32_t n_pages, int32_t flags);

/* Creates a paged context (arguments as ams_ctx_create, plus n_pages in
 * [0, batch * capacity / 64] and flags).  Errors: AMS_EINVAL, AMS_ENOMEM,
 * AMS_EHIP. */
ams_status ams_ctx_create_paged(ams_model* m, int32_t batch, int32_t capacity, int32_t max_pass_tokens,
                                int32_t n_pages, int32_t flags, void* ws, size_t ws_bytes, ams_ctx** out);

/* The page table (host int32 [batch][capacity / 64]: the pool page of each
 * row's 64-position block, -1 for a row that holds no pages: never built or
 * invalidated), the reference count of every pool page (host
 * int32 [n_pages]) and the number of pages in use; any output may be NULL.
 * A context created with ams_ctx_create keeps page b * capacity / 64 + i for
 * row b's block i and reports every page in use. */
ams_status ams_ctx_pages(const ams_ctx* c, int32_t* page_table, int32_t* refs, int32_t* pages_in_use);

/* Paper section 3.2.1 (Constructing the Action Context): the intermediate
 * state of an inference -- here every layer's K/V of the step-invariant prefix
 * -- is computed once and kept in the context pool for later inferences.
 *
 * Builds the context from each row's prefix: `prefix` is a device array
 * [sum_b lens[b]][d] in the model dtype, rows packed one after another
 * (row b's tokens at positions 0..lens[b]-1); `lens` is a host array [batch]
 * with 1 <= lens[b] <= capacity.  Computes and keeps every layer's K/V
 * and the final hidden state of each row's last token.  Any previous
 * content is discarded.  State -> READY.
 * Errors: AMS_EINVAL, AMS_ECAPACITY, AMS_EHIP. */
ams_status ams_ctx_build(ams_ctx* c, const void* prefix, const int32_t* lens, void* stream);

/* Paper section 3.2.1: a later inference reuses the cached state instead of
 * recomputing it, and after the inference the unseen K/V (here the new
 * observation tokens') is added to the context.
 *
 * One action step.
 *   new_tokens: device [sum_b new_lens[b]][d] (model dtype) or NULL;
 *   new_lens:   host [batch] (0 allowed per row) or NULL for no new tokens.
 * The new tokens are appended to the rows' contexts first (their K/V kept:
 * the paper's post-inference insert).  Then n_actions bins are decoded
 * greedily per row: the first from the last committed token's hidden state,
 * each later one after feeding back the previous bin's embedding (vocabulary
 * id vocab - n_bins + bin).  The fed-back tokens occupy scratch positions
 * that are dropped when the call ends, so committed lengths grow only by
 * new_lens.  Ties between equal logits go to the lowest bin.
 *   out_tokens: device int32 [batch][n_actions]: chosen bins.
 *   out_logits: device fp32 [batch][n_actions][n_bins] or NULL.
 *   forced:     device int32 [batch][n_actions] or NULL: when given, bin
 *               forced[b][j] is fed back after action j instead of the
 *               argmax (teacher forcing); out_tokens still reports the
 *               argmax.  Forced bins are clamped into [0, n_bins).
 * Requires READY (else AMS_ESTATE), 1 <= n_actions, and for every row
 * len[b] + new_lens[b] + n_actions - 1 <= capacity (else AMS_ECAPACITY).
 * Errors: AMS_EINVAL, AMS_ESTATE, AMS_ECAPACITY, AMS_EHIP. */
ams_status ams_ctx_step(ams_ctx* c, const void* new_tokens, const int32_t* new_lens,
                        int32_t n_actions, int32_t* out_tokens, float* out_logits,
                        const int32_t* forced, void* stream);

/* Paper section 3.3 (Handler, common part): on an exception the current
 * slice is discarded and the next inference starts from freshly collected
 * environment data -- the caller then rebuilds from the new prefix.
 *
 * Discards the context (host-side only; enqueues nothing).  State -> INVALID;
 * lengths read 0 until the next build. */
ams_status ams_ctx_invalidate(ams_ctx* c);

/* Paper section 3.3 (Handler, common part) applied to one robot of a batch:
 * the exception handler discards that episode's slice and re-infers from
 * freshly collected environment data while the other episodes' contexts stay
 * as they are (section 4 keeps this control on the CPU).
 *
 * Rebuilds only the listed rows: `rows` is a host array of n_rows strictly
 * increasing row indices, `prefix` a device array [sum_i lens[i]][d] of their
 * new prefixes packed in that order, `lens` a host array [n_rows] with
 * 1 <= lens[i] <= capacity.  The listed rows' K/V, last hidden state and
 * length are replaced; every other row is untouched.  Rows may be READY,
 * INVALID or EMPTY; the context is READY once every row is.
 * Errors: AMS_EINVAL, AMS_ECAPACITY, AMS_EHIP. */
ams_status ams_ctx_build_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, const void* prefix,
                              const int32_t* lens, void* stream);

/* Paper section 3.3 (Handler, common part), one robot of a batch: discards
 * the listed rows' contexts (host-side only; enqueues nothing).  `rows` as for
 * ams_ctx_build_rows.  Those rows read length 0 and the context is INVALID
 * (no ams_ctx_step) until each of them is rebuilt with ams_ctx_build_rows;
 * the other rows keep their contexts.  Errors: AMS_EINVAL. */
ams_status ams_ctx_invalidate_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows);

/* Paper section 3.2.1 (the post-inference insert on its own): appends new
 * observation tokens to the rows' contexts (their K/V kept, lengths grow by
 * new_lens) without decoding actions -- the first half of ams_ctx_step.
 *   new_tokens: device [sum_b new_lens[b]][d] (model dtype);
 *   new_lens:   host [batch], 0 allowed per row.
 * Requires READY (else AMS_ESTATE) and len[b] + new_lens[b] <= capacity for
 * every row (else AMS_ECAPACITY).  Errors: AMS_EINVAL, AMS_ESTATE,
 * AMS_ECAPACITY, AMS_EHIP. */
ams_status ams_ctx_append(ams_ctx* c, const void* new_tokens, const int32_t* new_lens, void* stream);

/* Paper section 3.2.2 (Layered Storage of Action Context): rarely used
 * context moves from GPU memory to CPU memory and back.
 *
 * Bytes of the host image of a row of `len` positions (0 if len is outside
 * [1, capacity]): a 256-byte header, every layer's K and V of the row's
 * positions ([layer][K|V][head][len][head_dim] in the compute type: fp16 for
 * bf16 models, fp32 otherwise), the last position's hidden state (fp32 [d])
 * and its fp16 pair ([d] + [d]). */
size_t ams_ctx_row_host_bytes(const ams_ctx* c, int32_t len);

/* Copies each listed row's context (READY rows; strictly increasing indices)
 * into host[i]: pinned host memory (hipHostMalloc, mapped), 16-byte aligned,
 * at least ams_ctx_row_host_bytes(c, row length) bytes, caller-owned.  The
 * library's kernels write the images through the buffers' device addresses
 * (the header is written by the host at once).  The rows become OFFLOADED
 * (length 0, not steppable; the context reads INVALID) and, in a paged
 * context, their pages return to the pool; later work on the same stream
 * may reuse them.  The images are complete once the stream has passed the
 * call.  Errors: AMS_EINVAL, AMS_ESTATE, AMS_EHIP. */
ams_status ams_ctx_offload_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, void* const* host, void* stream);

/* Restores rows from host images written by ams_ctx_offload_rows (of a
 * context of the same model; host[i] as there): rows[i] gets the image's
 * context -- every layer's K/V, its length and last hidden state -- on fresh
 * pages of a paged context, and is READY afterwards.  A listed row must not be
 * READY.  Errors: AMS_EINVAL (not an image of this model), AMS_ESTATE,
 * AMS_ECAPACITY (image longer than the capacity, or not enough free pages:
 * nothing changed), AMS_EHIP. */
ams_status ams_ctx_reload_rows(ams_ctx* c, const int32_t* rows, int32_t n_rows, const void* const* host,
                               void* stream);

/* Each row's state into host array states[batch]: 0 EMPTY, 1 READY,
 * 2 INVALID, 3 OFFLOADED. */
ams_status ams_ctx_row_states(const ams_ctx* c, int32_t* states);

/* Paper sections 3.2.2 (Layered Storage of Action Context) and 3.2.3 (Auto
 * Eviction): which rows to evict from the GPU to free pages_needed pages.
 * Host-only arithmetic over host arrays [n_rows]: priority (lower goes
 * first), last_use (a tick of the caller's, larger = more recent), pages held,
 * droppable (nonzero: the caller keeps the row's inputs, so dropping and
 * recomputing it is allowed), resident (nonzero: on the GPU), pinned (nonzero:
 * never evicted).  The resident unpinned rows are taken in increasing
 * (priority, last_use, row) order until the pages taken reach pages_needed;
 * action[r] = 0 keep, 1 offload to host memory (ams_ctx_offload_rows), 2 drop
 * (ams_ctx_invalidate_rows, later ams_ctx_build_rows).  *pages_freed (may be
 * NULL) receives the pages the taken rows hold, less than pages_needed when
 * the candidates hold fewer.  Errors: AMS_EINVAL. */
ams_status ams_tier_plan(int32_t n_rows, const int32_t* priority, const int64_t* last_use, const int32_t* pages,
                         const int32_t* droppable, const int32_t* resident, const int32_t* pinned,
                         int64_t pages_needed, int32_t* action, int64_t* pages_freed);

/* Paper section 3.2.1 (the diffusion model's latent vectors are cached action
 * context) and section 3.4.2 (Action Regeneration: generation starts from a
 * stored successful latent instead of noise): a flow-matching action head over
 * the cached context.  Each row's action chunk is a latent of n_tokens tokens
 * of action_dim values.  The velocity runs every decoder layer over the tokens
 * W_in x_i + tau w_t at the positions right after the row's committed
 * sequence (causal attention over the cache and the earlier chunk tokens;
 * their K/V are scratch, the context is unchanged), then reads out
 * W_out (h_i / rms(h_i)) (rms with the model's epsilon, no gain).
 * Weights in the model dtype: w_in [d][action_dim], w_t [d],
 * w_out [action_dim][d], device, caller-owned. */
typedef struct {
  const void *w_in, *w_t, *w_out;
  int32_t action_dim; /* 1..256 */
  int32_t n_tokens;   /* >= 1 */
} ams_flow_head;

/* Euler integration of every row's latent from tau0 (in [0, 1)) to 1 in
 * n_steps equal steps, in place: x is device fp32 [batch][n_tokens][action_dim]
 * holding the initial latents (noise for a cold start at tau0 = 0, a stored
 * latent for a warm start at a later tau0) and receiving the final ones.
 * Requires READY and len[b] + n_tokens <= capacity for every row.
 * Errors: AMS_EINVAL, AMS_ESTATE, AMS_ECAPACITY, AMS_EHIP. */
ams_status ams_ctx_flow(ams_ctx* c, const ams_flow_head* head, float* x, float tau0, int32_t n_steps,
                        void* stream);

/* Committed length of every row into host array lens[batch]. */
ams_status ams_ctx_lengths(const ams_ctx* c, int32_t* lens);

/* Current state: 0 EMPTY, 1 READY, 2 INVALID; negative status on error. */
int32_t ams_ctx_state(const ams_ctx* c);

/* 1 when this context's action decode (everything ams_ctx_step does after
 * appending new tokens) runs as one persistent launch, 0 when it runs as a
 * sequence of per-layer kernels; negative status on error.  The persistent
 * launch serves bf16 models with up to 8 rows (environment AMS_FUSED=0 at
 * context creation turns it off); it keeps one workgroup per compute unit
 * resident and synchronises them between the layers' phases, so it assumes
 * no other work holds the compute units meanwhile.  Should the device not keep
 * them all resident, its bounded waits give up, every out_tokens entry of that
 * step reads -1 (never a valid bin), and the next ams_ctx_step on the context
 * returns AMS_EHIP with the context INVALID (ams_ctx_state reads INVALID as
 * soon as the failed launch has ended; ams_ctx_build recovers). */
int32_t ams_ctx_persistent_decode(const ams_ctx* c);

#ifdef __cplusplus
}
#endif

#endif /* AMS_H */
