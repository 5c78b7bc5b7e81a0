/*
 * kvr.h - budgeted in-place KV-cache repair on one MI355X (gfx950) GPU.
 *
 * The method (paper, Section 3 "Cache Repair as Budgeted Recomputation"):
 * a context C of n tokens has been prefilled into a key/value cache K(C).  A
 * contiguous, length-preserving edit turns C into C' (c_i = c'_i outside the
 * half-open span S = [edit_start, edit_end)), so positions and rotary phases
 * are unchanged.  Repair recomputes a position set P = S u A, where A holds K
 * positions chosen downstream of the span, from C' layer by layer over the
 * stale cache and leaves every other cache entry unchanged ("The repair
 * interface").  Recomputing every position reproduces the full prefill
 * K(C') (Eq. 1).
 *
 * The model is a Llama-style pre-norm decoder: RMSNorm, Q/K/V projections
 * (optional bias), rotary embedding (rotate-half pairing, angle
 * p * theta^(-2i/head_dim) at each token's absolute position p), causal
 * grouped-query attention with scale 1/sqrt(head_dim), output projection,
 * SwiGLU MLP, residual connections and a final RMSNorm.
 *
 * Conventions for every call
 * - All calls return kvr_status; no C++ exception crosses this interface.
 * - Pointers named d_* are device pointers (hipMalloc'd or equivalent) on the
 *   context's device; h_* are host pointers.  The caller owns every buffer it
 *   passes; the library never frees them.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).  GPU
 *   work is enqueued on it and the call returns without waiting; outputs are
 *   valid once the stream has reached that point.  Calls on one context use
 *   the context's workspace and must be ordered (one stream, or synchronised
 *   by the caller); one context per host thread.
 * - Arguments are validated before anything is enqueued: on any status other
 *   than KVR_OK or KVR_E_HIP, no GPU work was enqueued and no cache was
 *   touched.  KVR_E_HIP means a HIP call failed after enqueueing began; cache
 *   contents are then undefined.  kvr_last_error() describes the failure.
 *
 * Data layouts
 * - Weights: dtype of kvr_dims.dtype (fp32 or bf16), row-major.  Linear
 *   weights are [out_features][in_features]; norm gains and biases are
 *   vectors.  All weight pointers must be 16-byte aligned.
 * - KV cache of one document: [n_layers][2][n_kv_heads][n_cap][head_dim]
 *   (index 0 = keys after rotary embedding, 1 = values), dtype of
 *   kvr_dims.dtype, 16-byte aligned.  kvr_cache_bytes() gives its size.
 * - Tokens: int32 ids in [0, vocab).
 * - Hidden outputs: fp32 rows of d_model values = the final RMSNorm output.
 */
#ifndef KVR_H
#define KVR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KVR_OK = 0,
    KVR_E_ARG = 1,          /* NULL pointer, bad dims, unsorted/duplicate positions ... */
    KVR_E_RANGE = 2,        /* a size or position outside what the call allows */
    KVR_E_UNSUPPORTED = 3,  /* a shape or dtype this build does not handle */
    KVR_E_NOMEM = 4,        /* workspace allocation failed */
    KVR_E_HIP = 5           /* a HIP runtime call or kernel launch failed */
} kvr_status;

typedef enum { KVR_F32 = 0, KVR_BF16 = 1 } kvr_dtype;

/* Model and workspace dimensions.
 * head_dim must be even and at most 128; n_heads a multiple of n_kv_heads.
 * d_model must be a multiple of 4 and at most 16384, and the fused
 * projection width (n_heads + 2 n_kv_heads) * head_dim a multiple of 4;
 * other shapes give KVR_E_UNSUPPORTED.
 * max_ctx bounds n_cap of every cache the context is used with (it sizes the
 * rotary table); max_rows bounds the total number of repaired rows |P| summed
 * over the documents of one kvr_repair call.  fp32 computes every step in
 * fp32; bf16 keeps weights, cache and matrix operands in bf16 with fp32
 * accumulation, fp32 softmax/RMSNorm and an fp32 residual stream. */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
    int32_t qkv_bias;      /* 1: Q/K/V projections carry a bias */
    float rms_eps;
    double rope_theta;
    int32_t max_ctx;
    int32_t max_rows;
    kvr_dtype dtype;
} kvr_dims;

/* Device pointers of one layer.  wq [n_heads*head_dim][d_model],
 * wk/wv [n_kv_heads*head_dim][d_model], wo [d_model][n_heads*head_dim],
 * w_gate/w_up [d_ffn][d_model], w_down [d_model][d_ffn], attn_norm/mlp_norm
 * [d_model]; bq/bk/bv are NULL unless qkv_bias. */
typedef struct {
    const void *attn_norm, *wq, *wk, *wv, *bq, *bk, *bv, *wo;
    const void *mlp_norm, *w_gate, *w_up, *w_down;
} kvr_layer_weights;

/* embed [vocab][d_model] and final_norm [d_model] on the device; `layers` is a
 * HOST array of n_layers entries (copied by kvr_create); lm_head
 * [vocab][d_model] is the output projection used only by kvr_score and
 * kvr_generate (NULL: tied to embed). */
typedef struct {
    const void *embed, *final_norm;
    const kvr_layer_weights *layers;
    const void *lm_head;
} kvr_weights;

typedef struct kvr_ctx kvr_ctx;

/* Create a context on the current HIP device.  The weight pointers are
 * borrowed (not copied) and must stay valid until kvr_destroy.  The context
 * allocates its workspace (sized from max_rows, max_ctx and the model dims),
 * a pinned host staging buffer and, in bf16, a copy of every projection
 * matrix and of the LM head repacked in MFMA operand order (about the size of
 * the model's matrices); kvr_workspace_bytes reports the device total.
 * Errors: KVR_E_ARG (NULL/invalid dims or misaligned/missing weights),
 * KVR_E_UNSUPPORTED, KVR_E_NOMEM, KVR_E_HIP.  On error *out is NULL and the
 * message is available through kvr_last_error(NULL). */
kvr_status kvr_create(const kvr_dims *dims, const kvr_weights *weights, kvr_ctx **out);

/* Release the workspace.  Waits for the context's outstanding work. NULL ok. */
void kvr_destroy(kvr_ctx *ctx);

/* Bytes of one document's cache: n_layers*2*n_kv_heads*n_cap*head_dim*elem. */
size_t kvr_cache_bytes(const kvr_dims *dims, int32_t n_cap);

/* Device bytes held by the context (workspace, rotary table, scratch). */
size_t kvr_workspace_bytes(const kvr_ctx *ctx);

/* Full prefill K(C) (Section 3, "Question Setting"): run the decoder over all
 * n tokens of d_tokens, writing the keys/values of positions [0, n) of every
 * layer into d_cache (slots >= n are not touched).  If d_hidden_out is not
 * NULL it receives the final RMSNorm output of every position, [n][d_model]
 * fp32.  1 <= n <= n_cap <= max_ctx. */
kvr_status kvr_prefill(kvr_ctx *ctx, const int32_t *d_tokens, int32_t n, int32_t n_cap,
                       void *d_cache, float *d_hidden_out, void *stream);

/* One document of a repair call. */
typedef struct {
    void *d_cache;              /* stale cache K(C), updated in place */
    int32_t n, n_cap;           /* context length and the cache's slot capacity */
    const int32_t *d_tokens_new;/* the full edited context C' [n] (device) */
    int32_t edit_start, edit_end; /* half-open span S, 0 <= start <= end <= n */
    const int32_t *h_positions; /* A: strictly ascending, in [0, n), disjoint
                                   from S (host; copied during the call) */
    int32_t n_positions;
    float *d_hidden_out;        /* [|P|][d_model] fp32 rows in ascending
                                   position order, or NULL */
} kvr_doc;

/* Repair R(K(C), C', P) with P = [edit_start, edit_end) u h_positions for each
 * document (paper Section 3, "The repair interface").  Layer by layer, the
 * rows of P are recomputed from C' (their embeddings at layer 0, their own
 * outputs of the previous layer above it); at each layer the fresh keys and
 * values of all of P are written into the cache first, then every p in P
 * attends over slots t <= p of its own document, fresh where t is in P and
 * stale elsewhere.  Slots outside P are never written.  Upstream positions
 * (< edit_start) are accepted (the full-position endpoint, Eq. 1, needs
 * them); policies select only downstream positions (kvr_select).
 * Documents are independent; they are batched into one pass per layer, so
 * their caches must not overlap (the byte ranges [d_cache, d_cache +
 * kvr_cache_bytes(n_cap)) of the documents with a non-empty P are disjoint).
 * A document with an empty span and no positions is a no-op.
 * Errors: KVR_E_ARG (NULL pointers, unsorted/duplicate positions, positions
 * inside the span, overlapping caches), KVR_E_RANGE (span or position outside [0, n), n > n_cap,
 * n_cap > max_ctx, sum of |P| > max_rows). */
kvr_status kvr_repair(kvr_ctx *ctx, const kvr_doc *docs, int32_t n_docs, void *stream);

typedef enum { KVR_EDIT_LOCAL = 0, KVR_RANDOM = 1 } kvr_policy;

/* Host-only position selection (paper Table 1; no context, no device).
 * The pool is D = [edit_end, n - 1).  EDIT_LOCAL returns the first
 * min(K, |D|) positions of D.  RANDOM returns min(K, |D|) distinct positions
 * drawn uniformly from D: a SplitMix64 generator (Steele, Lea and Flood,
 * OOPSLA 2014) seeded with `seed` drives a partial Fisher-Yates shuffle of D
 * in ascending order, j = i + next() mod (|D| - i) for i < K, and the first
 * entries are returned sorted ascending.  h_out must hold K entries; *n_out
 * receives the count.  Errors: KVR_E_ARG (NULL outputs, K < 0, bad policy),
 * KVR_E_RANGE (n < 1 or not 0 <= edit_start <= edit_end <= n). */
kvr_status kvr_select(kvr_policy policy, int32_t n, int32_t edit_start, int32_t edit_end,
                      int32_t K, uint64_t seed, int32_t *h_out, int32_t *n_out);

/* Fresh-query forward and teacher-forced scoring over a (repaired) cache
 * (Section 3, "What counts as repaired": the margin m_x is the difference of
 * the length-averaged teacher-forced log-probabilities of two answers; Eq. 2
 * and Eq. 3 are computed from it and from kvr_generate).  The m tokens
 * d_tokens[n .. n+m) are appended after the n cached positions: they run
 * through the decoder attending over cache rows [0, n) and causally over each
 * other, their keys/values are written into cache slots [n, n+m) (scratch:
 * rows [0, n) are not touched), and the LM head and a log-softmax over the
 * vocabulary follow.  Outputs (device): for j < m-1,
 *   d_logprob[j] = log p(d_tokens[n+j+1] | d_tokens[0 .. n+j]),
 * and for j < m, d_argmax[j] = the most probable token after position n+j
 * (lowest id among equal maxima); d_argmax may be NULL, d_logprob may be NULL
 * only when m == 1.  Errors: KVR_E_ARG (NULL context, cache or tokens,
 * misaligned cache), KVR_E_RANGE (not 0 <= n, 1 <= m, n + m <= n_cap <=
 * max_ctx, or m above the context's pass size), KVR_E_NOMEM (the first call
 * allocates the scoring buffers), KVR_E_HIP. */
kvr_status kvr_score(kvr_ctx *ctx, void *d_cache, int32_t n, int32_t n_cap, const int32_t *d_tokens, int32_t m,
                     float *d_logprob, int32_t *d_argmax, void *stream);

/* Greedy continuation (the generation y_b of Eq. 3): appends the q query
 * tokens d_tokens[n .. n+q) after the n cached positions as kvr_score does,
 * then generates max_new tokens one at a time, each the most probable token
 * after the previous one (lowest id among equal maxima), and writes them to
 * d_tokens[n+q .. n+q+max_new).  The whole loop is enqueued on `stream`: each
 * generated id is written on the device and read by the next step's forward.
 * Cache slots [n, n+q+max_new-1) are scratch.  Errors as kvr_score, with
 * KVR_E_RANGE unless 1 <= q, 1 <= max_new and n + q + max_new - 1 <= n_cap. */
kvr_status kvr_generate(kvr_ctx *ctx, void *d_cache, int32_t n, int32_t n_cap, int32_t *d_tokens, int32_t q,
                        int32_t max_new, void *stream);

/* Repair metrics on the host (Section 3, "What counts as repaired"; no
 * context, no device).  For a cache state x the margin m_x is the
 * length-averaged teacher-forced log-probability of the post-edit answer
 * minus that of the pre-edit answer.
 *
 * kvr_answer_logprob: the mean log-probability of the answer_len answer
 * tokens of a block scored by kvr_score as query_len query tokens followed by
 * the answer; h_logprob is kvr_score's d_logprob copied to the host
 * (n_logprob entries; entry j predicts appended token j+1, so the answer is
 * predicted by entries query_len-1 .. query_len+answer_len-2).
 * Errors: KVR_E_ARG (NULL), KVR_E_RANGE (query_len < 1, answer_len < 1, or
 * the answer not inside the block). */
kvr_status kvr_answer_logprob(const float *h_logprob, int32_t n_logprob, int32_t query_len, int32_t answer_len,
                              double *out);

/* Eq. 2, margin recovery (unclipped): *out = (m_repaired - m_stale) /
 * (m_oracle - m_stale) and *defined = 1, or *out = 0 and *defined = 0 when the
 * stale-to-oracle gap is zero (such items are left out of the mean).
 * Errors: KVR_E_ARG (NULL outputs). */
kvr_status kvr_margin_recovery(double m_repaired, double m_stale, double m_oracle, double *out, int32_t *defined);

/* Eq. 3 for one item: *out = 1 when the post-edit answer h_a_new occurs in the
 * greedy continuation (from kvr_generate) as a contiguous token run and the
 * pre-edit answer h_a_old does not, else 0; the flip rate is the mean over
 * the retained items.  An empty answer occurs in every continuation.
 * Errors: KVR_E_ARG (NULL array with a positive length, negative lengths,
 * NULL out). */
kvr_status kvr_flipped(const int32_t *h_continuation, int32_t n_continuation, const int32_t *h_a_new, int32_t n_new,
                       const int32_t *h_a_old, int32_t n_old, int32_t *out);

/* CacheBlend selector (Table 1: top-K by the key/value deviation of one early
 * layer; Section 3, "Cost accounting": about one prefill layer over the
 * changed suffix).  Runs the positions [edit_start, n) of C' (d_tokens_new,
 * n ids) through layers 0 .. layer-1 and the key/value projection of `layer`
 * into a context-owned scratch copy (the stale cache d_cache is only read;
 * its rows before edit_start stand in for the fresh ones, which the edit
 * cannot change), then for every pool position p in D = [edit_end, n - 1)
 *   dev = ||K_fresh[p] - K_stale[p]||_2 + ||V_fresh[p] - V_stale[p]||_2
 * (norms over all kv heads and dimensions of `layer`), and writes to d_out
 * (device, K entries) the min(K, |D|) positions of largest deviation (ties:
 * lower position) in ascending order; *n_out (host) receives that count.  The
 * paper's "layer 2" is layer = 1 (counting from one).  d_dev_out (device,
 * |D| floats, or NULL) receives the deviations of D in position order.
 * Errors: KVR_E_ARG (NULL argument, negative K, misaligned cache),
 * KVR_E_RANGE (bad n/n_cap/span or layer), KVR_E_NOMEM, KVR_E_HIP. */
kvr_status kvr_select_cacheblend(kvr_ctx *ctx, const void *d_cache, int32_t n, int32_t n_cap,
                                 const int32_t *d_tokens_new, int32_t edit_start, int32_t edit_end, int32_t K,
                                 int32_t layer, int32_t *d_out, float *d_dev_out, int32_t *n_out, void *stream);

/* Attention selector (Table 1: top-K by the query's attention over the stale
 * cache; Section 3, "Cost accounting": one stale-cache scoring pass).  Runs
 * the q query tokens d_tokens[n .. n+q) after the n stale positions of
 * d_cache, as kvr_score does (they attend over the stale cache and causally
 * over each other; their keys/values land in cache slots [n, n+q), which are
 * scratch; rows [0, n) are only read), and accumulates for every stale
 * position p < n
 *   mass[p] = sum over layers, query heads and query tokens of the softmax
 *             probability that the token places on p
 * (the aggregation rule is a reading: the paper does not state it).  Writes to
 * d_out (device, K entries) the min(K, |D|) positions of the pool
 * D = [edit_end, n - 1) with the largest mass (ties: lower position) in
 * ascending order; *n_out (host) receives that count.  d_mass_out (device,
 * n floats, or NULL) receives mass[0 .. n).  d_tokens must hold n + q ids
 * (only the query's are read).  The last layer's output projection and MLP
 * are not run: the mass is complete after its attention.
 * Errors: KVR_E_ARG (NULL argument, negative K, misaligned cache),
 * KVR_E_RANGE (need 1 <= n, 1 <= q <= the context's rows per pass,
 * n + q <= n_cap <= max_ctx, 0 <= edit_start <= edit_end <= n),
 * KVR_E_NOMEM, KVR_E_HIP. */
kvr_status kvr_select_attention(kvr_ctx *ctx, void *d_cache, int32_t n, int32_t n_cap, const int32_t *d_tokens,
                                int32_t q, int32_t edit_start, int32_t edit_end, int32_t K, int32_t *d_out,
                                float *d_mass_out, int32_t *n_out, void *stream);

/* kvr_select_attention for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, semantics and errors as kvr_select_attention,
 * with the selector's scratch (the per-kv-head mass [n_kv_heads][n], the
 * query rows' log-sum-exp [q][n_heads] and, when d_mass_out is NULL, the mass
 * [n]; each part rounded up to 256 bytes) in a fixed device array of
 * 4 MiB (4194304 bytes) that the library holds on each device it runs on
 * until the process ends, instead of a context buffer grown on first use.
 * Nothing is allocated on the device or the host heap (with the step
 * profiler off; kvr_create allocated the context beforehand).  Every call on
 * one device shares that array: calls that overlap in time on one device
 * (two streams, two contexts, two threads) race and give undefined results;
 * calls ordered on one stream are independent (nothing in the array needs to
 * start at zero).  Additional errors: KVR_E_RANGE when the scratch above
 * exceeds 4 MiB (about n_kv_heads * n <= 1,000,000 with d_mass_out given);
 * KVR_E_HIP if the array's device address could not be obtained. */
kvr_status kvr_select_attention_noalloc(kvr_ctx *ctx, void *d_cache, int32_t n, int32_t n_cap,
                                        const int32_t *d_tokens, int32_t q, int32_t edit_start, int32_t edit_end,
                                        int32_t K, int32_t *d_out, float *d_mass_out, int32_t *n_out, void *stream);

/* EditLocal@boundary (Section 5.2, "How Far the Window Should Extend"): the
 * structural variant that recomputes from the end of the edit to the next
 * document boundary, with no selector forward.  Returns the positions
 * [edit_end, min(boundary, n - 1)) of the pool D = [edit_end, n - 1) in
 * ascending order; `boundary` is the position where the next document
 * begins (boundary == edit_end selects nothing).  h_out must hold `capacity`
 * entries.  Errors: KVR_E_ARG (NULL outputs or capacity < 0), KVR_E_RANGE
 * (n < 1, not 0 <= edit_start <= edit_end <= n, boundary < edit_end, or more
 * than `capacity` positions; nothing is written then). */
kvr_status kvr_select_to_boundary(int32_t n, int32_t edit_start, int32_t edit_end, int32_t boundary,
                                  int32_t capacity, int32_t *h_out, int32_t *n_out);

/* Transplant (Section 3, "Transplant is not recomputation"): copy the key and
 * value rows of the given positions, every layer and kv head, from d_src (for
 * the diagnostic: the oracle cache K(C')) into d_dst (the stale cache).  A
 * localization diagnostic that needs the oracle cache, not a repair method.
 * Both caches use the layout of kvr_prefill with their own n_cap; positions
 * (host array, copied during the call) must lie in [0, min(src_n_cap,
 * dst_n_cap)) and be strictly ascending.  Enqueued on `stream` as device
 * copies, one per run of consecutive positions.  Errors: KVR_E_ARG (NULL
 * context or caches, unsorted positions, misaligned caches), KVR_E_RANGE
 * (a position out of range), KVR_E_HIP. */
kvr_status kvr_transplant(kvr_ctx *ctx, const void *d_src, int32_t src_n_cap, void *d_dst, int32_t dst_n_cap,
                          const int32_t *h_positions, int32_t n_positions, void *stream);

/* Per-step GPU time accounting, a tracing aid for benchmarks.  While enabled
 * (it is off after kvr_create), every kernel launch of a prefill or repair
 * pass is made with a pair of HIP events that the dispatch records at the
 * start and at the end of the kernel's execution (hipExtLaunchKernel), tagged
 * with the step of the layer loop it belongs to ("embed", "rmsnorm",
 * "qkv_proj", "rope_scatter", "attention", "attention_combine", "o_proj",
 * "gate_up_swiglu", "down_proj", "final_norm", and for the scoring calls
 * "lm_head", "logsoftmax").  The time of a launch is its
 * execution time; the dispatch gaps between kernels are not counted, so the
 * step times sum to less than the pass.  Errors: KVR_E_ARG (NULL context). */
kvr_status kvr_profile_enable(kvr_ctx *ctx, int32_t enable);

/* Wait for the recorded events, add their times to per-step totals and report
 * them: for i < min(*n_steps, capacity), names[i] (static strings), total_ms[i]
 * and launches[i] accumulated since the previous read; the totals are then
 * cleared.  *n_steps receives the number of steps.  Errors: KVR_E_ARG (NULL
 * context, n_steps or, when capacity > 0, output arrays), KVR_E_HIP. */
kvr_status kvr_profile_read(kvr_ctx *ctx, int32_t capacity, const char **names, double *total_ms,
                            int64_t *launches, int32_t *n_steps);

/* Text of the last failure on this context, or of the last failed
 * kvr_create/kvr_select when ctx is NULL.  Never NULL; valid until the next
 * call on the same context. */
const char *kvr_last_error(const kvr_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* KVR_H */
