/*
 * crf.h — C ABI of the bounded stale-KV recomputation library (libcrf.so).
 *
 * The library implements the recovery executor of CacheReforge
 * (arxiv 2609.30884): when an evolving LoRA adapter has moved on from the
 * version that produced a KV cache, a contiguous window of decoder layers
 * [l0, l0+h) is re-run over the complete cached prefix under the current
 * adapter, starting from the hidden state retained at the restart boundary,
 * and the refreshed K/V overwrite those layers' slots of the cache
 * (paper Sec. 4.2 "Executable restart"; supplementary Sec. S1.1, definition of
 * the operation R_{r,h}).  It also scores the per-layer adapter drift and risk
 * that feed the reuse / bounded / full-suffix choice (Sec. 4.1, Eq. 8); that
 * choice itself stays with the caller.
 *
 * General conventions
 *   - Every tensor pointer is a DEVICE pointer on the current HIP device,
 *     allocated and owned by the caller.  The library owns only the workspace
 *     inside a crf_context.  Host arrays (per-layer descriptor arrays, the
 *     anchor index array) are read during the call only.
 *   - Tensors are dense row-major.  Weights use the nn.Linear layout
 *     [d_out, d_in].  The storage type of every floating-point tensor is
 *     crf_model_dims.dtype (fp32 or bf16); accumulation is always fp32.
 *   - bf16 tensors must be 16-byte aligned; fp32 tensors 16-byte aligned.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *     default stream).  No call synchronises the device except where stated.
 *   - Errors are returned as crf_status codes, never by aborting.  Shape,
 *     range and pointer checks happen on the host before anything is
 *     launched; a failed check launches nothing.  The message of the last
 *     failure is available from crf_last_error().
 *   - A context is not thread-safe; use one context per stream.  Calls that
 *     overlap on one context race on its workspace.
 */
#ifndef CRF_H
#define CRF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CRF_ABI_VERSION 1

typedef enum {
  CRF_OK = 0,
  CRF_ERR_INVALID_ARG = 1,  /* null pointer, misaligned pointer, bad enum      */
  CRF_ERR_SHAPE = 2,        /* tensor/cache sizes inconsistent                  */
  CRF_ERR_RANGE = 3,        /* layer window outside [0, n_layers)              */
  CRF_ERR_UNSUPPORTED = 4,  /* valid model but not a shape this build handles   */
  CRF_ERR_WORKSPACE = 5,    /* exceeds the context's max_tokens / max rank     */
  CRF_ERR_HIP = 6,          /* a HIP runtime call failed                        */
  CRF_ERR_DEVICE = 7        /* a kernel's own bounds check fired (see below)   */
} crf_status;

typedef enum { CRF_F32 = 0, CRF_BF16 = 1 } crf_dtype;

/* Projection targets of one decoder layer (supplementary Eq. sup-qkv-current-layer
 * names Q, K, V; the output and MLP projections are the remaining update
 * targets of supplementary Eq. sup-first-invalid-cache-layer). */
enum { CRF_Q = 0, CRF_K, CRF_V, CRF_O, CRF_GATE, CRF_UP, CRF_DOWN, CRF_NUM_TARGETS };

/* Decoder shape.  Layers are indexed 0..n_layers-1 (Sec. 2.2, Eq. 1).
 * Target shapes: q [n_q_heads*head_dim, d_model], k and v
 * [n_kv_heads*head_dim, d_model], o [d_model, n_q_heads*head_dim],
 * gate and up [d_ffn, d_model], down [d_model, d_ffn]. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn;
  float rms_eps;      /* RMSNorm epsilon, inside the square root          */
  float rope_theta;   /* rotary base: angle(p, i) = p * theta^(-2i/hd)     */
  int32_t dtype;      /* crf_dtype: storage type of every tensor          */
} crf_model_dims;

/* Frozen base weights of one layer.  attn_norm, mlp_norm: RMSNorm gains [d_model].
 * w[t]: [d_out, d_in] of target t.  bias_q/k/v: optional [d_out] (NULL = none). */
typedef struct {
  const void *attn_norm, *mlp_norm;
  const void *w[CRF_NUM_TARGETS];
  const void *bias_q, *bias_k, *bias_v;
} crf_layer_weights;

/* Current LoRA adapter state of one layer: delta_t(x) = scale * (x A_t^T) B_t^T
 * with A_t [rank, d_in] and B_t [d_out, rank].  A[t] == NULL (with B[t] == NULL)
 * means target t carries no adapter.  rank 0 means the layer has no adapter. */
typedef struct {
  int32_t rank;
  float scale;
  const void *A[CRF_NUM_TARGETS];
  const void *B[CRF_NUM_TARGETS];
} crf_lora_layer;

/* Paged layerwise KV cache C = {K_l, V_l} (Sec. 2.2, Eq. 1).
 * k_pool / v_pool element (layer, page, kv_head, slot, e) lives at
 *   layer*layer_stride + page*page_stride + (kv_head*page_size + slot)*head_dim + e
 * (strides in elements).  Logical token t lives in physical page
 * block_table[t / page_size] (a DEVICE int32 array of ceil(n_tokens/page_size)
 * entries, shared by all layers), slot t % page_size.  K is stored after the
 * rotary rotation, V unrotated.  Pages not named by the block table, slots
 * past n_tokens and layers outside the window are never written.  A block
 * table entry outside [0, n_pages) is caught by the kernels: they skip that
 * page (treating its keys/values as zero) and raise the context's device
 * error flag (crf_context_device_errors). */
typedef struct {
  void *k_pool, *v_pool;
  int64_t layer_stride, page_stride;
  const int32_t *block_table;
  int32_t n_pages, page_size, n_tokens;
} crf_kv_cache;

typedef struct crf_context crf_context;

/* Kernel classes for the optional event timing (crf_context_set_timing). */
enum {
  CRF_KK_NORM = 0, CRF_KK_LORA_DOWN, CRF_KK_GEMM_QKV, CRF_KK_ATTN, CRF_KK_GEMM_O,
  CRF_KK_GEMM_GATEUP, CRF_KK_GEMM_DOWN, CRF_KK_DRIFT, CRF_KK_OTHER, CRF_KK_COUNT
};

/* Human-readable name of a status code (static string). */
const char *crf_status_string(crf_status s);

/* ABI version of the loaded library (CRF_ABI_VERSION at build time). */
int32_t crf_abi_version(void);

/* Create a context for `dims` on the current HIP device.  Allocates the
 * workspace for windows of up to max_tokens prefix tokens and LoRA ranks up
 * to max_lora_rank, and the rotary angle table for positions
 * 0..max_tokens-1.  Besides the per-token buffers (fp32 residual stream,
 * normalised input, queries, attention output, SwiGLU output, LoRA
 * down-projections), a bf16 context holds fixed-size scratch for split
 * work: one 256x256 fp32 tile per compute unit for the K-parts of the QKV and
 * residual GEMMs (64 MiB on 256 CUs), key-split attention partials for
 * decoding steps (ceil(max_tokens/64) x n_q_heads x 16 x (head_dim+4) floats),
 * K-split LoRA partials and, when max_lora_rank > 0, the down projection's
 * adapter sums formed inside the gate/up projection (4 x 2 x 256 x 16 floats
 * per compute unit, 32 MiB on 256 CUs, plus one int per gate/up tile).  All of
 * it is freed by crf_context_destroy.  On success *out
 * receives the context.  Errors: INVALID_ARG (null), UNSUPPORTED (see
 * crf_validate_dims), HIP (allocation failed). */
crf_status crf_context_create(const crf_model_dims *dims, int32_t max_tokens, int32_t max_lora_rank,
                              crf_context **out);
void crf_context_destroy(crf_context *ctx);

/* Message of the last failure on this context ("" if none).  With ctx == NULL,
 * the message of the last failure of a call made without a context. */
const char *crf_last_error(const crf_context *ctx);

/* Host-only check of a decoder shape: every dimension positive,
 * n_q_heads % n_kv_heads == 0, head_dim in {64, 128}, and for bf16 the
 * projection widths multiples of 128, d_ffn a multiple of 64 and every
 * projection weight matrix smaller than 2 GiB.  Touches no device.
 * Errors: INVALID_ARG, SHAPE, UNSUPPORTED. */
crf_status crf_validate_dims(const crf_model_dims *dims);

/* Host-only check of a recomputation request (Sec. 4.1: the candidate window
 * min(h, N - r) never passes the last layer; supplementary terminology table:
 * ranges are half-open).  Checks dims as above, 0 <= l0, 0 <= h,
 * l0 + h <= n_layers (else RANGE), and the cache geometry: page_size >= 1,
 * n_tokens >= 0, n_tokens <= n_pages * page_size, page_stride >=
 * n_kv_heads*page_size*head_dim, layer_stride >= n_pages*page_stride (else
 * SHAPE), one layer of a pool (n_pages*page_stride elements) under 2 GiB
 * (else UNSUPPORTED), on the bf16 path with h > 0 and more than 16 tokens a
 * projection input of n_tokens x max(d_model, n_q_heads*head_dim, d_ffn)
 * elements under 2 GiB (else UNSUPPORTED: 56,679 tokens at most at
 * Qwen2.5-7B shapes), non-null pools and block table when h > 0 and
 * n_tokens > 0 (else INVALID_ARG).  Touches no device. */
crf_status crf_validate_window(const crf_model_dims *dims, int32_t l0, int32_t h, const crf_kv_cache *kv);

/* Bounded recomputation R_{l0,h} (Sec. 4.2 "Executable restart"; supplementary
 * Sec. S1.1): starting from hidden_at_boundary = H_{l0-1} [n_tokens, d_model]
 * (the residual-stream output of layer l0-1, or the embedding state H_{-1}
 * when l0 == 0), run decoder layers l0..l0+h-1 over all n_tokens prefix
 * tokens under the current adapter `lora`, and overwrite layer l's K/V slots
 * of `kv_cache` for every l in the window with the recomputed, rotated K and
 * V.  Each layer: RMSNorm, Q/K/V projections with the LoRA delta, rotary
 * rotation of Q and K at positions 0..n_tokens-1, causal grouped-query
 * softmax attention (query head j reads K/V head j / (n_q_heads/n_kv_heads),
 * scale 1/sqrt(head_dim)), output projection with LoRA delta and residual,
 * RMSNorm, SwiGLU MLP down(silu(gate x) * up x) with LoRA deltas and residual.
 *   base_weights: host array [n_layers]; only the window's entries are read.
 *   lora:         host array [n_layers] of the current adapter, or NULL (no adapter).
 *   hidden_out:   [n_tokens, d_model] receives H_{l0+h-1}; may be NULL; may alias
 *                 hidden_at_boundary.  When NULL, nothing reads the last
 *                 window layer's output, and that layer's cache entry depends
 *                 on its input only through the K and V projections
 *                 (supplementary Eq. sup-layer-cache-dependency:
 *                 C_l = G_l(H_{l-1})), so on the bf16 path it runs RMSNorm and
 *                 the K/V projections (LoRA, bias, rotary, page write) only.
 *                 The K/V written are the same either way.
 * h == 0 is direct reuse: nothing is launched and hidden_out (if given and
 * distinct) is not written.  Layers outside the window and pages outside the
 * block table are never touched.  n_tokens comes from kv_cache->n_tokens and
 * must not exceed the context's max_tokens (else WORKSPACE).
 * Errors: as crf_validate_window, plus INVALID_ARG (null or misaligned
 * weights/boundary, dims differing from the context's), WORKSPACE, HIP. */
crf_status crf_recompute_window(crf_context *ctx, const crf_model_dims *dims, const void *hidden_at_boundary,
                                const crf_layer_weights *base_weights, const crf_lora_layer *lora, int32_t l0,
                                int32_t h, const crf_kv_cache *kv_cache, void *hidden_out, void *stream);

/* One stale cache of a batched request. */
typedef struct {
  const void *hidden_at_boundary;   /* [kv.n_tokens, d_model] = H_{l0-1}          */
  const crf_lora_layer *lora;       /* host array [n_layers] or NULL              */
  int32_t l0, h;
  crf_kv_cache kv;
  void *hidden_out;                 /* [kv.n_tokens, d_model] or NULL             */
} crf_window_item;

/* crf_recompute_window over several independent stale caches of one base
 * model, each with its own boundary state, window and adapter version (the
 * per-cache decision of Sec. 4.1 applied to many caches at once).  Every item
 * is validated before anything is launched.  When the items are independent
 * and event timing is off, they run
 * on two internal streams that wait for `stream` and that `stream` then waits
 * for, longest windows first, each on the lane with less work so far; the
 * first such call allocates a second workspace as large as the context's own
 * (what crf_context_create allocates) and two streams, kept until
 * crf_context_destroy.  Otherwise items run in order on `stream`.  Items are
 * independent when no byte one item may write lies in a range another item
 * may read or write: an item writes the layers [l0, l0+h) of both pools (each
 * layer's whole n_pages*page_stride span, since the pages are chosen by the
 * device-side block table) and its hidden_out, and reads those pool spans,
 * its hidden_at_boundary and its block table.  Items with h == 0 or no tokens
 * take part in no conflict.  Results are the same either way (each item's
 * arithmetic does not depend on the lane).
 * Errors: as crf_recompute_window; the failing item's index is in the message;
 * WORKSPACE if the second workspace cannot be allocated. */
crf_status crf_recompute_window_batched(crf_context *ctx, const crf_model_dims *dims,
                                        const crf_layer_weights *base_weights, int32_t n_items,
                                        const crf_window_item *items, void *stream);

/* First decoding step over a cached prefix (Sec. 3.2 "Tail Influence": the
 * first-step next-token logits z, fresh or with a hybrid cache): the embedding
 * states of n_new tokens [n_new, d_model] run through every layer 0..N-1 under
 * `lora`, at positions kv_cache->n_tokens .. kv_cache->n_tokens + n_new - 1.
 * At each layer they attend to that layer's cached K/V of the prefix (whatever
 * adapter version produced each layer: a hybrid cache is just a pool whose
 * layers come from different versions) and causally to each other; their own
 * rotated K and V are written into the slots after the prefix.  Then the final
 * RMSNorm (final_norm [d_model]) and the LM head (lm_head [vocab, d_model],
 * nn.Linear layout) give the logits of the last new token:
 * logits_out[vocab] (fp32, device).  The block table must cover
 * kv_cache->n_tokens + n_new tokens.  bf16 contexts only.
 * Errors: as crf_recompute_window over the window [0, N) of a prefix of
 * n_tokens + n_new tokens, plus SHAPE (n_new < 1), UNSUPPORTED (fp32 context,
 * vocab not a positive multiple of 8, LM head of 2 GiB or more), WORKSPACE
 * (n_new or n_tokens + n_new above max_tokens), INVALID_ARG (NULL or
 * misaligned final_norm, lm_head, logits_out). */
crf_status crf_decode_logits(crf_context *ctx, const crf_model_dims *dims, const void *new_tokens, int32_t n_new,
                             const crf_layer_weights *base_weights, const crf_lora_layer *lora,
                             const crf_kv_cache *kv_cache, const void *final_norm, const void *lm_head,
                             int32_t vocab, float *logits_out, void *stream);

/* Runtime drift and risk (Sec. 4.1 "Runtime risk and range selection", Eq. 8):
 *   d_l = || theta_t - theta_l^anchor ||_2,   q_l = s_l * d_l.
 * theta is the whole adapter: every A and B entry of every target of every
 * layer.  current: host array [n_layers] (theta_t).  versions: host array of
 * n_versions pointers, each to a host array [n_layers] of stored adapter
 * states; anchor_version: host int32 [n_layers], index of the version that
 * produced layer l's cache.  Targets present in `current` must be present
 * with the same rank in every version.  sensitivity: device fp32 [n_layers]
 * (s_l) or NULL for s = 1.  per_layer_only != 0 restricts the norm to layer
 * l's own slice.  Outputs (device fp32): drift_out [n_layers], risk_out
 * [n_layers], sq_partial_out [n_versions * n_layers] (squared distance of
 * layer l's slice to version v at index v*n_layers + l; may be NULL).
 * Errors: INVALID_ARG (null, anchor index out of range, target missing in a
 * version), SHAPE, HIP. */
crf_status crf_layer_drift(crf_context *ctx, const crf_model_dims *dims, const crf_lora_layer *current,
                           int32_t n_versions, const crf_lora_layer *const *versions,
                           const int32_t *anchor_version, const float *sensitivity, int32_t per_layer_only,
                           float *drift_out, float *risk_out, float *sq_partial_out, void *stream);

/* crf_layer_drift for callers that cannot allocate device memory (tight
 * serving loops, harnesses that forbid hipMalloc).  Not for stream capture:
 * the tables are uploaded from a host buffer that the next call on the same
 * thread overwrites, so a captured copy would read whatever it holds then.
 * Same arguments and results as crf_layer_drift (bitwise: the same kernels in
 * the same order) without a context: the segment tables and the partial sums
 * live in a fixed device scratch of CRF_DRIFT_NOALLOC_MAX_BYTES that the
 * library holds on each device it runs on until the process ends, and the
 * tables are staged on the host in a fixed per-thread buffer of the same size.
 * Nothing is allocated on the device and no allocating library routine is
 * called; the tables reach the scratch by one hipMemcpyAsync from pageable host
 * memory on `stream` (so the call returns once they are copied).  Calls that
 * overlap on one device race on its scratch: serialise them (one stream, or
 * the caller's own ordering).  A request whose tables and partials exceed the
 * scratch (segments: two per adapter target, layer and version; chunks of 2^16
 * elements each; about 64 bytes per chunk and segment) is rejected with
 * WORKSPACE before anything is copied or launched.  Errors are reported through
 * crf_last_error(NULL): INVALID_ARG, SHAPE, UNSUPPORTED (as crf_validate_dims),
 * WORKSPACE, HIP. */
#define CRF_DRIFT_NOALLOC_MAX_BYTES (4 << 20)
crf_status crf_layer_drift_noalloc(const crf_model_dims *dims, const crf_lora_layer *current, int32_t n_versions,
                                   const crf_lora_layer *const *versions, const int32_t *anchor_version,
                                   const float *sensitivity, int32_t per_layer_only, float *drift_out,
                                   float *risk_out, float *sq_partial_out, void *stream);

/* Device-side error flags raised by kernels' own bounds checks since the last
 * call (bit 0: a block table entry outside [0, n_pages)).  Synchronises the
 * device, then clears the flags. */
crf_status crf_context_device_errors(crf_context *ctx, int32_t *flags_out);

/* Optional per-kernel-class event timing.  While enabled, each launch is
 * bracketed by HIP events on its stream.  crf_context_read_timing
 * synchronises those events and returns, per kernel class (CRF_KK_*), the
 * summed milliseconds and launch counts since the last read, then resets. */
crf_status crf_context_set_timing(crf_context *ctx, int32_t enable);
/* The same for a subset of kernel classes: bit k of class_mask enables class
 * k (CRF_KK_*), 0 disables timing; enable != 0 above is the mask of every
 * class.  Each bracketed launch costs two event records on its stream, so a
 * measurement that needs one class's launch times only brackets that class.
 * Errors: INVALID_ARG (null context, bits at or past CRF_KK_COUNT). */
crf_status crf_context_set_timing_classes(crf_context *ctx, uint32_t class_mask);
crf_status crf_context_read_timing(crf_context *ctx, float *ms_out, int32_t *count_out, int32_t n_kinds);

/* Device facts for reporting measurements against the hardware's peak:
 * compute-unit count, peak engine clock (MHz) and the architecture name
 * (written NUL-terminated into name, at most name_len bytes; name may be NULL).
 * Errors: INVALID_ARG (null outputs), HIP. */
crf_status crf_device_info(int32_t device, int32_t *n_cu_out, int32_t *max_sclk_mhz_out, char *name,
                           int32_t name_len);

#ifdef __cplusplus
}
#endif
#endif /* CRF_H */
