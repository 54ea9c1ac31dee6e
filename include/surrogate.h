/*
 * surrogate.h - C ABI of the batched forecast-scoring library (libsurrogate.so).
 *
 * The library scores forecast queries with a dense decoder-only transformer in a
 * prefill-only pass on one MI355X (gfx950).  A query is the tokenized prompt of
 * x_i = (reference kernel, candidate kernel, hardware) from Section 2.1 of the paper
 * (Forecasting Relative Performance).  At the last prompt position the model's
 * next-token log-probabilities of a fixed set of verdict tokens give a forecast
 * distribution p_i, a predicted verdict (argmax) and a confidence q_i = max_b p_{i,b}
 * (Section 2.1).  Selective use (Section 2.1, Selective Use; budgeted measurement in
 * Section 3.1) then splits a batch into forecasts to accept and candidates to defer
 * to GPU measurement.  With the paper's eight speedup bins (Table 3) the forecast head
 * also gives each candidate an expected speedup, by which a search measures only the
 * best-ranked candidates (Sections 3.1 and 3.5), and discovery scores Pr[g >= x]
 * (Section 3.6).
 *
 * Conventions shared by every call:
 *  - Every call returns a surrogate_status; 0 is success, negative values are errors.
 *    On error, surrogate_last_error() returns a thread-local description.
 *  - Pointers suffixed _d are device pointers, _h host pointers.  The caller owns every
 *    buffer it passes; the library keeps no pointer to them after the call returns
 *    (device work stays stream-ordered: buffers must stay valid until the stream has
 *    passed the call's work).
 *  - Device work is enqueued on the caller's stream and is asynchronous.  Host-checkable
 *    argument errors are reported synchronously and then nothing is enqueued.
 *  - A model handle is read-only after loading; concurrent calls on one handle are
 *    allowed only with distinct workspaces and output buffers.
 *  - A call that fails after it took device memory releases it before returning, and a
 *    failed scoring, prefix or cache call leaves the model and its caches as they were
 *    (a failed cache_extend leaves its entries at their previous lengths).  For testing
 *    these paths, the environment variable SURROGATE_FAULT=alloc:N makes the N-th device
 *    or pinned allocation of a call fail (SURR_E_OOM) and SURROGATE_FAULT=launch:N the
 *    N-th checked HIP call of a call (SURR_E_HIP), counted from 1 in each call that loads
 *    weights, builds prefixes, creates a cache or scores (score_pairs, score_suffixes,
 *    cache_extend), each of which re-reads the variable; no other call is affected.
 */
#ifndef SURROGATE_H
#define SURROGATE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SURR_OK = 0,
    SURR_E_INVALID_ARG = -1, /* null pointer, bad count, bad mode, bad threshold/budget */
    SURR_E_SHAPE = -2,       /* config shape unsupported, or a length outside [1, limit] */
    SURR_E_TOKEN_RANGE = -3, /* a token id outside [0, vocab) was seen on the device   */
    SURR_E_OOM = -4,         /* device or pinned host allocation failed                  */
    SURR_E_HIP = -5,         /* a HIP runtime call failed                                */
    SURR_E_WEIGHTS = -6,     /* weight tensor list or weight file does not match the config */
    SURR_E_WORKSPACE = -7,   /* workspace smaller than surrogate_workspace_size()        */
    SURR_E_IO = -8           /* weight file cannot be opened or read                     */
} surrogate_status;

typedef enum { SURR_F32 = 0, SURR_BF16 = 1 } surrogate_dtype;

typedef enum {
    SURR_SELECT_THRESHOLD = 0,
    SURR_SELECT_BUDGET = 1,
    SURR_SELECT_TOP_SCORE = 2
} surrogate_select_mode;

typedef struct surrogate_model surrogate_model; /* opaque: device weights + RoPE table */

/* opaque: keys and values of every layer for a set of shared prompt prefixes */
typedef struct surrogate_prefix_cache surrogate_prefix_cache;

/* Architecture of the decoder: pre-norm RMSNorm, rotate-half RoPE, causal grouped-
 * query attention (query head a reads kv head floor(a * n_kv_heads / n_q_heads)),
 * SwiGLU MLP, final RMSNorm and an untied LM head, no biases.
 * dtype selects the storage and GEMM-input type of the matrices (SURR_F32 or
 * SURR_BF16); norm gains are always float32.  Supported shapes: head_dim in
 * {32, 64, 128}; d_model, d_ff and head_dim*n_q_heads multiples of 64 (bf16) or of 32
 * (f32); n_q_heads a multiple of n_kv_heads; max_pos >= 1. */
typedef struct {
    int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab, max_pos;
    float rope_base, rms_eps;
    int32_t dtype;
} surrogate_config;

/* Load a model from a weight file (the surrogate of Section 2.1 is a language model prompted
 * with the forecast query; here a dense decoder with the architecture above).  The file is
 * little-endian:
 *   bytes [0, 8)        the magic "SURRWGT1";
 *   bytes [8, 16)       uint64 H, the length of the JSON header that follows;
 *   bytes [16, 16 + H)  the header, ASCII JSON:
 *     {"format": "surrogate-weights", "version": 1,
 *      "config": {"n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ff",
 *                 "vocab", "max_pos", "rope_base", "rms_eps": numbers,
 *                 "dtype": "bf16" | "f32"},
 *      "tensors": [{"name": .., "dtype": .., "shape": [rows, cols] ([cols] for norms),
 *                   "offset": ..}, ...]};
 *   each tensor's bytes at its offset, a multiple of 4096, tensors in the order below and
 *   not overlapping (bf16 as raw 16-bit patterns, f32 as IEEE floats, row-major).
 * Tensor order and names: embed [V, d]; per layer l: layers.l.attn_norm [d],
 * layers.l.w_qkv [d_q + 2 d_kv, d] (rows: q heads, then k heads, then v heads),
 * layers.l.w_o [d, d_q], layers.l.mlp_norm [d], layers.l.w_gate [d_ff, d],
 * layers.l.w_up [d_ff, d], layers.l.w_down [d, d_ff]; final_norm [d]; lm_head [V, d].
 * Norms are f32; matrices have the config's dtype.  Matrices are [out, in], so both
 * operands of every projection are contiguous along the reduction.
 * The whole header is checked before any device work (names, order, dtypes, shapes,
 * alignment, bounds).  The file is mapped read-only and copied into the model's device
 * arena; `stream` is synchronized before returning.
 * Errors: SURR_E_INVALID_ARG (nulls), SURR_E_IO (cannot open or map the file),
 * SURR_E_WEIGHTS (malformed header or tensors outside the file), SURR_E_SHAPE (config not
 * supported), SURR_E_OOM, SURR_E_HIP. */
surrogate_status surrogate_load_weights(const char *path, hipStream_t stream, surrogate_model **out);

/* The configuration a weight file declares, after the same checks surrogate_load_weights
 * makes on its header and table; no device work (usable without a GPU).
 * Errors: SURR_E_INVALID_ARG, SURR_E_IO, SURR_E_WEIGHTS. */
surrogate_status surrogate_weight_file_config(const char *path, surrogate_config *out);

/* Number of weight tensors surrogate_load_weights_tensors takes for cfg: 3 + 9 * n_layers. */
surrogate_status surrogate_tensor_count(const surrogate_config *cfg, int32_t *n_out);

/* Shape and element type of tensor `index` of surrogate_load_weights_tensors, in the order
 *   embed[V, d];
 *   per layer: attn_norm[d], w_q[d_q, d], w_k[d_kv, d], w_v[d_kv, d], w_o[d, d_q],
 *              mlp_norm[d], w_gate[d_ff, d], w_up[d_ff, d], w_down[d, d_ff];
 *   final_norm[d]; lm_head[V, d]
 * (d_q = n_q_heads * head_dim, d_kv = n_kv_heads * head_dim).  Matrices are row-major
 * [out, in]; norms are reported as rows = 1.  *dtype_out is SURR_F32 for norms and
 * cfg->dtype for matrices (bf16 = raw 16-bit patterns). */
surrogate_status surrogate_tensor_shape(const surrogate_config *cfg, int32_t index,
                                        int64_t *rows, int64_t *cols, int32_t *dtype_out);

/* As surrogate_load_weights from tensors already in memory, for callers that hold the
 * weights (tests, benchmarks) rather than a file: n_tensors = surrogate_tensor_count()
 * tensors in the order above; tensors[i] points to a dense row-major tensor of
 * surrogate_tensor_shape(i); all of them are host memory if tensors_on_device == 0, device
 * memory otherwise.  The library copies them into its own device arena (re-laid out for its
 * kernels: bf16 projection matrices are stored in 256-row panels of 256 x 32 blocks, each
 * placed through a transient device staging buffer of the largest matrix's size that is
 * freed before returning), builds the RoPE cos/sin table in float64 and stores it as
 * float32, and synchronizes `stream` before returning, so the sources may be freed
 * afterwards.
 * Errors: SURR_E_INVALID_ARG (nulls), SURR_E_SHAPE (unsupported config),
 * SURR_E_WEIGHTS (n_tensors mismatch), SURR_E_OOM, SURR_E_HIP. */
surrogate_status surrogate_load_weights_tensors(const surrogate_config *cfg,
                                                const void *const *tensors, int32_t n_tensors,
                                                int32_t tensors_on_device, hipStream_t stream,
                                                surrogate_model **out);

surrogate_status surrogate_get_config(const surrogate_model *m, surrogate_config *out);

/* Device workspace (bytes) that surrogate_score_pairs needs for a batch of `batch`
 * prompts holding `total_tokens` tokens in all, none longer than `max_len`. */
surrogate_status surrogate_workspace_size(const surrogate_model *m, int32_t batch,
                                          int64_t total_tokens, int32_t max_len, size_t *bytes);

/* Score a ragged batch (the prefill-only surrogate call).
 *  tokens_d      device int32 [batch, row_stride]; row i holds prompt i in its first
 *                lengths_h[i] entries; entries beyond are never read.
 *  lengths_h     host int32 [batch]; 1 <= lengths_h[i] <= min(row_stride, max_pos).
 *  verdict_ids_h host int32 [n_verdict], 1 <= n_verdict <= 16, distinct ids in [0, vocab).
 *  workspace_d   device buffer, 256-byte aligned, of workspace_bytes bytes.  With at least
 *                surrogate_workspace_size(m, batch, sum of lengths, max length) bytes the
 *                batch runs as one pass.  A smaller workspace (a token budget) makes the
 *                call score consecutive chunks of whole prompts, each the longest run of
 *                prompts that fits; outputs are the same, since a prompt's outputs do not
 *                depend on the other prompts.  The least workable size is that of the
 *                longest prompt alone, surrogate_workspace_size(m, 1, L, L).
 * Outputs (device, caller-owned):
 *  logprobs_d    float [batch, n_verdict]: log-softmax over the full vocabulary of the
 *                next-token logits at position lengths_h[i] - 1, at the verdict ids.
 *  probs_d       float [batch, n_verdict] or NULL: p_i = softmax of those log-probs.
 *  confidence_d  float [batch]: q_i = max_b p_{i,b}.
 *  verdict_d     int32 [batch] or NULL: argmax_b p_{i,b}, lowest index on ties.
 * A token id outside [0, vocab) is read as id 0 and raises a sticky device error that
 * surrogate_device_status() reports as SURR_E_TOKEN_RANGE.  Results are deterministic:
 * a prompt's outputs do not depend on the other prompts of the batch or on the run.
 * Errors (synchronous, nothing enqueued): SURR_E_INVALID_ARG, SURR_E_SHAPE,
 * SURR_E_WORKSPACE (a prompt alone does not fit), SURR_E_OOM (pinned staging), SURR_E_HIP. */
surrogate_status surrogate_score_pairs(surrogate_model *m, const int32_t *tokens_d,
                                       int64_t row_stride, const int32_t *lengths_h,
                                       int32_t batch, const int32_t *verdict_ids_h,
                                       int32_t n_verdict, void *workspace_d,
                                       size_t workspace_bytes, float *logprobs_d, float *probs_d,
                                       float *confidence_d, int32_t *verdict_d,
                                       hipStream_t stream);

/* Shared prefixes.  In the paper's workload every candidate of a task is scored in a prompt
 * that starts with the same system prompt and the task's one reference kernel (Section 3.2:
 * each candidate is compared against its task's single reference) and ends with the
 * candidate kernel.  That prefix is computed once: surrogate_prefix_build runs the
 * decoder over n_prefix prefixes (laid out like the prompts of surrogate_score_pairs:
 * tokens_d [n_prefix, row_stride], lengths_h[g] in [1, min(row_stride, max_pos - 1)],
 * a workspace of surrogate_workspace_size(m, n_prefix, sum of lengths, max length)) and
 * keeps every layer's keys (after RoPE) and values in a new cache, which owns its device
 * memory (n_layers * 2 * sum_g roundup(lengths_h[g], 64) * d_kv elements of the model's
 * dtype; surrogate_prefix_cache_bytes reports it).  The cache is ready for use once
 * `stream` has passed the build's work; it is read-only afterwards.
 * Errors: SURR_E_INVALID_ARG, SURR_E_SHAPE, SURR_E_WORKSPACE, SURR_E_OOM, SURR_E_HIP. */
surrogate_status surrogate_prefix_build(surrogate_model *m, const int32_t *tokens_d,
                                        int64_t row_stride, const int32_t *lengths_h,
                                        int32_t n_prefix, void *workspace_d,
                                        size_t workspace_bytes, hipStream_t stream,
                                        surrogate_prefix_cache **out);

/* As surrogate_score_pairs for prompts that continue cached prefixes: prompt i is prefix
 * prefix_id_h[i] (or nothing, for -1) followed by its lengths_h[i] tokens in tokens_d.
 * Every output equals that of surrogate_score_pairs on the concatenated prompt, up to
 * rounding order.  Positions continue after the prefix, so prefix length + lengths_h[i]
 * <= max_pos.  Workspace: surrogate_workspace_size(m, batch, sum of lengths_h, max of
 * lengths_h), or less, down to the longest prompt alone (chunked as in
 * surrogate_score_pairs).  The cache must come from the same model.
 * Errors as surrogate_score_pairs; SURR_E_INVALID_ARG for a prefix id outside
 * [-1, n_prefix) or a cache of another model. */
surrogate_status surrogate_score_suffixes(surrogate_model *m, const surrogate_prefix_cache *cache,
                                          const int32_t *prefix_id_h, const int32_t *tokens_d,
                                          int64_t row_stride, const int32_t *lengths_h,
                                          int32_t batch, const int32_t *verdict_ids_h,
                                          int32_t n_verdict, void *workspace_d,
                                          size_t workspace_bytes, float *logprobs_d,
                                          float *probs_d, float *confidence_d, int32_t *verdict_d,
                                          hipStream_t stream);

/* Decode continuation.  A cache also holds growing token sequences: entries with a
 * reserved capacity whose keys and values are appended by prefill and decode steps.
 * surrogate_cache_create reserves n_entries entries of capacity_h[g] tokens (1 <=
 * capacity <= max_pos; rounded up to 64), all empty, in device memory the cache owns
 * (cleared; synchronous).  surrogate_cache_extend appends lengths_h[i] tokens (tokens_d
 * [batch, row_stride], device) to entry entry_ids_h[i] for every i, with positions
 * continuing the entry (length + lengths_h[i] <= min(capacity, max_pos); an entry at
 * most once per call): the tokens attend to everything the entry held before and
 * causally to each other, exactly as the same tokens at the end of one long prompt would.
 * A prefill passes a whole prompt; a decode step passes one token per sequence.  After
 * the last appended token of each entry it writes (device, caller-owned, either may be
 * NULL) next_token_d[i], the first argmax of the next-token distribution over the
 * vocabulary (greedy decoding), and target_logprob_d[i], its full-vocabulary log-softmax at
 * target_ids_h[i] (host; teacher forcing).  The entry lengths advance when the call
 * returns (the device work is stream-ordered behind it); surrogate_cache_lengths reads
 * them and surrogate_cache_reset empties entries for reuse.  Workspace:
 * surrogate_workspace_size(m, batch, sum of lengths_h, max of lengths_h).  A cache made
 * by surrogate_prefix_build is an ordinary cache whose entries are full; any cache can
 * serve as the prefixes of surrogate_score_suffixes.
 * Errors: SURR_E_INVALID_ARG (nulls, entry or target ids out of range, an entry twice,
 * a cache of another model), SURR_E_SHAPE (lengths past the capacity or max_pos),
 * SURR_E_WORKSPACE, SURR_E_OOM, SURR_E_HIP. */
surrogate_status surrogate_cache_create(surrogate_model *m, int32_t n_entries,
                                        const int32_t *capacity_h, surrogate_prefix_cache **out);
surrogate_status surrogate_cache_extend(surrogate_model *m, surrogate_prefix_cache *cache,
                                        const int32_t *entry_ids_h, const int32_t *tokens_d,
                                        int64_t row_stride, const int32_t *lengths_h,
                                        int32_t batch, const int32_t *target_ids_h,
                                        void *workspace_d, size_t workspace_bytes,
                                        int32_t *next_token_d, float *target_logprob_d,
                                        hipStream_t stream);
surrogate_status surrogate_cache_lengths(const surrogate_prefix_cache *cache, int32_t *lengths_h);
surrogate_status surrogate_cache_reset(surrogate_prefix_cache *cache, const int32_t *entry_ids_h,
                                       int32_t n);

/* Device bytes held by the cache. */
surrogate_status surrogate_prefix_cache_bytes(const surrogate_prefix_cache *cache, size_t *bytes);

/* Release the cache's device memory; pending work that reads it must have completed.
 * NULL is ignored. */
void surrogate_prefix_free(surrogate_prefix_cache *cache);

/* Selective deferral on a device score vector confidence_d[n], 1 <= n <= 65536.  The
 * first list ("defer") is always the set sent to measurement on the device.
 *  SURR_SELECT_THRESHOLD: accept i iff confidence[i] >= threshold in float32 (the
 *    convention s >= tau of Section 3.6); NaN is never accepted.  budget_k is ignored.
 *    With discovery scores (surrogate_forecast_head) as input, the accepted list is the
 *    set predicted to be discovery moments.
 *  SURR_SELECT_BUDGET: defer the min(budget_k, n) candidates of lowest confidence
 *    (Section 3.1 measures a budgeted subset); order is confidence ascending with NaN
 *    first, ties by ascending index, -0.0 == +0.0.  budget_k < 0 is an error.
 *  SURR_SELECT_TOP_SCORE: the vector holds expected speedups S_hat; defer (measure) the
 *    min(budget_k, n) candidates of highest score, the top-c% of Section 3.1 and the
 *    best quarter a search measures in Section 3.5; order is score descending with NaN
 *    last, ties by ascending index, -0.0 == +0.0.  budget_k < 0 is an error.
 * Outputs (device): defer_idx_d[n] and accept_idx_d[n] receive the ascending index
 * lists (entries past each count are left untouched); counts_d[2] = {n_defer,
 * n_accept}, which sum to n.  Bit-exact and deterministic. */
surrogate_status surrogate_select(const float *confidence_d, int32_t n,
                                  surrogate_select_mode mode, float threshold, int32_t budget_k,
                                  int32_t *defer_idx_d, int32_t *accept_idx_d, int32_t *counts_d,
                                  hipStream_t stream);

/* The speedup-bin forecast head on forecasts probs_d[n, n_bins] (device, row-major,
 * e.g. the probs_d of surrogate_score_pairs with one verdict token per bin).
 *  bin_values_h  host [n_bins]: representative speedup m_b of each bin (Table 3: the
 *                interior values are geometric bin centres; the open first and last bins
 *                take empirical means, which the caller supplies).
 *  bin_edges_h   host [n_bins - 1], positive, strictly increasing: bin b covers
 *                (edge[b-1], edge[b]], the first bin everything up to edge[0], the last
 *                everything above edge[n_bins - 2].  Read only if n_cutoffs > 0.
 *  cutoffs_h     host [n_cutoffs], each in [edge[0], edge[n_bins - 2]].
 * Outputs (device, either may be NULL):
 *  expected_speedup_d  float [n]: S_hat_i = sum_b p_{i,b} m_b (Section 3.1).
 *  discovery_d         float [n, n_cutoffs]: s_i = Pr[g >= x_c] under p_i (Section 3.6),
 *                      with each interior bin's mass spread log-uniformly over the bin;
 *                      a cutoff on an edge sums whole bins.
 * 1 <= n_bins <= 16, 0 <= n_cutoffs <= 8 (n_bins >= 2 when n_cutoffs > 0), n >= 0.
 * Computed in float32 with the per-bin weights formed in float64 on the host.
 * Errors (synchronous, nothing enqueued): SURR_E_INVALID_ARG for nulls, counts out of
 * range, non-finite values, unordered edges or a cutoff outside the edges; SURR_E_HIP. */
surrogate_status surrogate_forecast_head(const float *probs_d, int64_t n, int32_t n_bins,
                                         const double *bin_values_h, const double *bin_edges_h,
                                         const double *cutoffs_h, int32_t n_cutoffs,
                                         float *expected_speedup_d, float *discovery_d,
                                         hipStream_t stream);

/* Forecast quality against measured speedups, for batches of evaluation candidates or RL
 * rollouts.  probs_d [n, n_bins] are forecasts (device, row-major), speedup_d [n] the
 * measured speedups S_i = T_ref / T_i (device, finite and positive), 1 <= n <= 65536,
 * 2 <= n_bins <= 16; bin_values_h / bin_edges_h as in surrogate_forecast_head (bin b
 * covers (edge[b-1], edge[b]]; a speedup's bin counts the edges strictly below it).
 * budgets_h [n_budgets], 1 <= n_budgets <= 8, are fractions c in (0, 1]: the top
 * max(1, floor(c n)) candidates by expected speedup are measured (ties by index).
 * Outputs (device; the per-candidate ones may be NULL):
 *  bin_d     int32 [n]: the measured bin y_i.
 *  brier_d   float [n]: Brier(p_i, y_i) = 1/2 sum_b (p_{i,b} - 1[b = y_i])^2 (Section 2.2).
 *  crps_d    float [n]: CRPS = 1/(n_bins - 1) sum_{k < n_bins - 1} (F_k - 1[y_i <= k])^2.
 *  summary_d double [8 + n_budgets]: accuracy (mean of the correctness reward
 *            1[argmax p_i = y_i], first argmax), mean Brier, mean CRPS, mean
 *            r_corr + 1 - Brier, mean r_corr + 1 - CRPS (Section 2.2), ECE over ten
 *            confidence buckets (floor(10 q) in float32, q = 1 in the last), forecast
 *            error mean |m_{argmax} - S_i|, speedup recovered averaged over the budgets
 *            (percent), then speedup recovered at each budget (Section 3.1).
 * workspace_d: device, 256-byte aligned, >= surrogate_evaluate_workspace_size(n, n_budgets).
 * Sums are taken in float64 in a fixed order (deterministic).
 * Errors (synchronous): SURR_E_INVALID_ARG, SURR_E_WORKSPACE, SURR_E_HIP. */
surrogate_status surrogate_evaluate_workspace_size(int32_t n, int32_t n_budgets, size_t *bytes);
surrogate_status surrogate_evaluate(const float *probs_d, const float *speedup_d, int32_t n,
                                    int32_t n_bins, const double *bin_values_h,
                                    const double *bin_edges_h, const double *budgets_h,
                                    int32_t n_budgets, void *workspace_d, size_t workspace_bytes,
                                    int32_t *bin_d, float *brier_d, float *crps_d,
                                    double *summary_d, hipStream_t stream);

/* surrogate_evaluate without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, outputs, limits and errors as surrogate_evaluate; the
 * caller still provides every input and output buffer.  The workspace is a fixed scratch
 * array in device memory of 4.5 MiB (room for n = 65536 forecasts with 8 budgets), one per
 * device, held from the library's loading until the process ends; its device address is
 * looked up on the first call on each device.  The call allocates nothing: no hipMalloc,
 * hipFree or allocating library routine.  Calls on one device share that device's
 * scratch, so calls that overlap on one device (different streams, or threads) race and
 * must be serialized by the caller.  Nothing carries over between calls: every scratch
 * byte a call reads it first writes.  Errors: as surrogate_evaluate, and SURR_E_WORKSPACE
 * if a call would need more than the scratch holds. */
surrogate_status surrogate_evaluate_noalloc(const float *probs_d, const float *speedup_d, int32_t n,
                                            int32_t n_bins, const double *bin_values_h,
                                            const double *bin_edges_h, const double *budgets_h,
                                            int32_t n_budgets, int32_t *bin_d, float *brier_d,
                                            float *crps_d, double *summary_d, hipStream_t stream);

/* Synchronize `stream` and report (then clear) the sticky device error of the model:
 * SURR_E_TOKEN_RANGE if an out-of-range token id was seen since the last check. */
surrogate_status surrogate_device_status(surrogate_model *m, hipStream_t stream);

/* Measurement hook.  Kernel phases of surrogate_score_pairs, surrogate_prefix_build and
 * surrogate_score_suffixes: */
typedef enum {
    SURR_PHASE_EMBED = 0,     /* varlen token packing + embedding gather          */
    SURR_PHASE_RMSNORM,       /* RMSNorm over all tokens (attention, MLP)          */
    SURR_PHASE_GEMM_QKV,      /* fused QKV projection                              */
    SURR_PHASE_ROPE,          /* rotary embedding of q and k                       */
    SURR_PHASE_ATTENTION,     /* causal GQA prefill attention                      */
    SURR_PHASE_GEMM_O,        /* output projection + residual, all tokens          */
    SURR_PHASE_GEMM_GATE_UP,  /* gate/up projection + SwiGLU, all tokens           */
    SURR_PHASE_GEMM_DOWN,     /* down projection + residual, all tokens            */
    SURR_PHASE_LAST_ROWS,     /* final layer's row-pruned work + final RMSNorm     */
    SURR_PHASE_LM_HEAD,       /* last-position LM head GEMM                        */
    SURR_PHASE_LSE_VERDICT,   /* full-vocab log-softmax + verdict read-out         */
    SURR_PHASE_PREFIX_CAPTURE, /* surrogate_prefix_build: copy of each layer's K/V  */
    SURR_N_PHASES
} surrogate_phase;

/* While enabled (enable != 0), surrogate_score_pairs brackets every kernel launch with
 * a pair of HIP events on its stream.  surrogate_profile_collect synchronizes those
 * events, writes per-phase totals since the previous collect (ms_out[SURR_N_PHASES]
 * milliseconds, launches_out[SURR_N_PHASES] launch counts) and resets them.  Not for
 * concurrent use on one model.  Errors: SURR_E_INVALID_ARG, SURR_E_HIP. */
surrogate_status surrogate_profile_enable(surrogate_model *m, int32_t enable);
surrogate_status surrogate_profile_collect(surrogate_model *m, double *ms_out,
                                           int64_t *launches_out);

/* Release the model's device memory.  Pending work that uses the model must have
 * completed.  NULL is ignored. */
void surrogate_free(surrogate_model *m);

const char *surrogate_status_string(surrogate_status s);

/* Thread-local detail of the last failing call on this thread ("" if none). */
const char *surrogate_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SURROGATE_H */
