/* sd.h - C ABI of the MI355X self-speculative decoding library.
 *
 * Greedy self-speculative decoding (Draft & Verify, Zhang et al., arXiv
 * 2309.08168) of a LLaMA-style decoder at batch size 1 on one GPU:
 *   - draft: the model with a chosen set of attention / MLP sublayers
 *     bypassed decodes tokens one at a time, until K_max tokens are drafted
 *     or right after a token whose top-1 probability is below gamma
 *     (Sec. 3.2 Algorithm 2, Sec. 3.4);
 *   - verify: the full model scores the last committed token and all drafts
 *     in one forward; the longest matching prefix is kept and the model's
 *     own next token follows it (Algorithm 2).  The emitted tokens equal
 *     greedy autoregressive decoding (Algorithm 1).
 *
 * Conventions for every function:
 *   - returns SD_OK (0) or a negative sd_status; on failure nothing was
 *     enqueued unless the status is SD_ERR_DEVICE, and sd_last_error()
 *     returns a message for the calling thread;
 *   - no C++ exception crosses this boundary;
 *   - "device" pointers are HIP device allocations on the current device;
 *     "host" pointers are ordinary CPU memory;
 *   - a model and its caches are used by one host thread at a time; all
 *     GPU work runs on the stream given to sd_model_create, in order.
 */
#ifndef SD_H
#define SD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SD_OK = 0,
    SD_ERR_INVALID_ARG = -1, /* a null pointer, a size out of range, a token id outside [0, vocab) */
    SD_ERR_CAPACITY = -2,    /* the KV cache cannot hold the requested positions */
    SD_ERR_OOM = -3,         /* a device or host allocation failed */
    SD_ERR_DEVICE = -4,      /* a HIP call or a kernel failed; the stream may hold partial results */
    SD_ERR_UNIMPLEMENTED = -5
} sd_status;

typedef enum { SD_F32 = 0, SD_BF16 = 1 } sd_dtype;

/* Model shape (the LLaMA-2 family the paper evaluates, Sec. 4.1).
 * d_model and ffn_dim are multiples of 8; head_dim is a power of two in
 * [16, 128]; n_heads is a multiple of n_kv_heads (grouped-query attention
 * when they differ).  dtype is the storage type of every weight
 * and of the KV cache; activations and accumulations are float32. */
typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    float rms_eps;   /* RMSNorm epsilon */
    float rope_base; /* rotary base; rotate-half pairing (i, i + head_dim/2) */
    sd_dtype dtype;
} sd_config;

/* Weights: DEVICE pointers in dtype, row-major [out, in] like nn.Linear.
 * Borrowed, never copied or freed ("no extra memory": the draft model is
 * the same weights with sublayers bypassed, Sec. 3.2); they must outlive
 * the model.  The per-layer members are HOST arrays of n_layers device
 * pointers, copied at create time.
 *   tok_emb   [vocab, d]            final_norm [d]     lm_head [vocab, d]
 *   attn_norm [d]                   mlp_norm   [d]
 *   w_qkv     [(n_heads + 2 n_kv_heads) head_dim, d]: q rows, k rows, v rows
 *   w_o       [d, n_heads head_dim]
 *   w_gate_up [2 ffn, d]: ffn gate rows, then ffn up rows
 *   w_down    [d, ffn]
 * Every device pointer must be 16-byte aligned. */
typedef struct {
    const void *tok_emb, *final_norm, *lm_head;
    const void *const *attn_norm, *const *w_qkv, *const *w_o;
    const void *const *mlp_norm, *const *w_gate_up, *const *w_down;
} sd_weights;

typedef struct sd_model sd_model;
typedef struct sd_kv_cache sd_kv_cache;

/* Statistics of one generate call.  stage_log, when not NULL, is a HOST
 * array of stage_log_cap (k_e, n_e) pairs: drafts and accepted drafts of
 * each stage in order (entries past stage_log_cap are dropped). */
typedef struct {
    int64_t n_stages;      /* draft/verify stages (0 for autoregressive) */
    int64_t n_drafted;     /* sum of k_e */
    int64_t n_accepted;    /* sum of n_e; acceptance rate = n_accepted / n_drafted */
    int64_t n_emitted;     /* tokens written to out_tokens */
    int64_t n_draft_steps; /* draft forwards run */
    double prefill_ms;     /* prompt forward, GPU time */
    double draft_ms;       /* all draft forwards, GPU time */
    double verify_ms;      /* all verification forwards (with acceptance), GPU time */
    double decode_ms;      /* GPU time from the end of prefill to the last token */
    double total_ms;       /* GPU time of the whole call */
    int32_t *stage_log;
    int32_t stage_log_cap;
    float *gamma_log;      /* HOST float [stage_log_cap] or NULL: the threshold each stage drafted with */
    /* Self-speculative calls enqueue the first part of the next step ahead,
     * on a prediction of the device's decision, so that the GPU does not
     * wait for the host between steps; a part the decision does not confirm
     * is cancelled on the device (its kernels return at once). */
    int64_t n_guarded_noop_steps; /* parts enqueued ahead and cancelled */
    double noop_ms;               /* their GPU time; decode_ms - draft_ms - verify_ms - noop_ms is the
                                   * time the GPU waited for the host */
} sd_stats;

/* Parameters of the adaptive draft exit (Sec. 3.4, Eqs. 2-4).  After every
 * verification stage e with k_e > 0 drafts, AR <- beta1 AR + (1 - beta1) AR_e
 * with AR_e = n_e / k_e (AR = AR_e at the first such stage); the threshold
 * moves to gamma + epsilon when AR <= alpha and to gamma - epsilon otherwise,
 * smoothed: gamma <- beta2 gamma + (1 - beta2) (gamma +- epsilon).  The
 * update runs in float64 in that order; the exit test compares the top-1
 * probability with the threshold rounded to float32.  The paper's settings:
 * gamma0 0.6, epsilon 0.01, beta1 0.5, beta2 0.9, alpha 0.70-0.90. */
typedef struct {
    double gamma0, alpha, epsilon, beta1, beta2;
} sd_adaptive;

/* Creates a model over borrowed device weights.  hip_stream is a
 * hipStream_t (NULL = the default stream).  Validates the shape and
 * allocates the library's device workspace (activations of up to 16 rows,
 * rotary table, reduction scratch; for bfloat16 models with head_dim 32, 64
 * or 128 also the large-forward workspace of 1024 rows, about 270 MB at the
 * 13B shape).  Errors: INVALID_ARG, OOM, DEVICE. */
sd_status sd_model_create(const sd_config *config, const sd_weights *weights, void *hip_stream, sd_model **out);
/* Waits for the model's stream, then frees the model and its workspace.
 * KV caches created on it stay valid objects but are detached: they can
 * only be destroyed (any other use reports INVALID_ARG). */
sd_status sd_model_destroy(sd_model *model);

/* Bytes of a KV cache for capacity positions:
 * n_layers * 2 * n_kv_heads * capacity * head_dim * sizeof(dtype). */
size_t sd_kv_cache_bytes(const sd_config *config, int32_t capacity);

/* KV caches.  Both decoding stages attend over the cache of the tokens so
 * far (Sec. 3.2): the draft of the full model's prefix, the verification of
 * the committed prefix plus the drafts it scores in one forward; rejected
 * drafts are rolled back by truncation (Algorithm 2).
 *
 * Creates a KV cache of capacity positions (1..65536), length 0.  device_buf, when
 * not NULL, is a caller-owned device buffer of sd_kv_cache_bytes() bytes
 * (borrowed), laid out [n_layers][2 (K, V)][n_kv_heads][capacity][head_dim]
 * in the model dtype, with rotary position embedding already applied to K;
 * otherwise the library allocates it.  Errors: INVALID_ARG, CAPACITY
 * (more than 65536 positions), OOM. */
sd_status sd_kv_cache_create(sd_model *model, int32_t capacity, void *device_buf, sd_kv_cache **out);
/* Frees the cache (and its buffer when the library allocated it), after
 * waiting for its model's stream; allowed before or after sd_model_destroy. */
sd_status sd_kv_cache_destroy(sd_kv_cache *cache);
int32_t sd_kv_cache_length(const sd_kv_cache *cache); /* -1 for NULL */
/* Rolls the cache back to len positions (0 <= len <= length). */
sd_status sd_kv_cache_truncate(sd_kv_cache *cache, int32_t len);
/* Declares positions [0, len) valid, for caches the caller filled itself
 * (0 <= len <= capacity). */
sd_status sd_kv_cache_set_length(sd_kv_cache *cache, int32_t len);

/* The decoder forward of both stages (Sec. 3.2): with skip_mask the draft
 * model, which bypasses the chosen attention and MLP sublayers (Sec. 3.3),
 * without it the original model, which verifies several tokens in one
 * forward (Algorithm 2).
 *
 * One forward of n tokens (HOST int32 [n], each in [0, vocab)) at positions
 * [len, len + n) of cache; writes K/V of every attention sublayer that
 * skip_mask keeps and sets len += n.  skip_mask is a HOST uint8
 * [2 n_layers] (entry 2l: attention of layer l, 2l+1: its MLP; 1 = bypass,
 * i.e. the identity on the residual stream) or NULL for the full model.
 * logits, when not NULL, is a DEVICE float32 [n, vocab].  More than 16
 * rows on a model with the large-forward workspace run in chunks of up to
 * 1024 rows on matrix-core GEMMs (the prompt prefill of the generate calls
 * takes the same path); otherwise rows run in chunks of at most 16.
 * Errors: INVALID_ARG, CAPACITY (nothing enqueued), DEVICE. */
sd_status sd_forward(sd_model *model, const int32_t *tokens, int32_t n, const uint8_t *skip_mask,
                     sd_kv_cache *cache, float *logits);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * forward as sd_forward for n <= 16 rows, with identical results, calling no
 * hipMalloc, hipFree or other allocating routine and copying nothing from
 * host memory (the tokens travel as a kernel argument).  Its scratch
 * (activations, split partials, attention partials, lm-head partials, the
 * control block) lives in a static device array of 32 MiB that each GPU the
 * library runs on holds until the process ends; a model and cache capacity
 * that need more are refused (over 4096 positions the 13B shape needs about
 * 28 MiB, the 70B shape 30 MiB).  Every call on one GPU shares that GPU's
 * array: calls that overlap on one GPU (other streams, other threads, other
 * models) race and must not be made.  The model's workspace and the cache
 * are the caller's, created beforehand (those calls allocate); the call
 * waits for its stream like sd_forward.  Errors: INVALID_ARG (also n > 16),
 * CAPACITY (cache full, or scratch above 32 MiB; nothing enqueued), DEVICE. */
sd_status sd_forward_static(sd_model *model, const int32_t *tokens, int32_t n, const uint8_t *skip_mask,
                            sd_kv_cache *cache, float *logits);

/* FP8 draft weights.  The adaptation appendix (Quantization subsection and
 * table) combines self-speculative decoding with FP8 and FP4 weights to cut
 * memory.  Here only a copy of the draft's weights is quantized, so that a
 * draft step streams one byte per weight; the verification keeps the
 * stored bf16 weights, so the emitted tokens are still exactly those of
 * greedy decoding of the original model (only drafts and stage traces
 * follow the copy).  This trades the "no extra memory" property of the
 * plain draft for speed: one byte per quantized weight and four bytes per
 * row.
 *
 * Quantizes the QKV, output, gate/up and down weights of every sublayer
 * skip_mask (HOST, layout of sd_forward) keeps to OCP FP8 E4M3 with one
 * power-of-two scale 2^e per output row (e the smallest integer with
 * max|W[n][:]| 2^-e <= 448; each byte the nearest E4M3 value of
 * W[n][k] 2^-e, ties to even).  From then on every one-row forward with a
 * skip mask (the draft steps of the generate calls, sd_forward of one row
 * with a mask) reads the copy of each sublayer that has one; forwards
 * without a mask read the bf16 weights, and sd_forward refuses masked
 * forwards of more than one row.  skip_mask NULL removes the copies.
 * bfloat16 models only.  Errors: INVALID_ARG, OOM, DEVICE. */
sd_status sd_model_quantize_draft(sd_model *model, const uint8_t *skip_mask);
/* The FP8 copy of (layer, kind), kind 0 QKV, 1 output, 2 gate/up, 3 down:
 * DEVICE bytes [N][K] and exponents int32 [N], or NULL when the sublayer
 * has none (for inspection). */
sd_status sd_model_draft_fp8(const sd_model *model, int32_t layer, int32_t kind, const void **q,
                             const int32_t **exps);

/* Greedy self-speculative decoding (Algorithm 2, static gamma exit of
 * Sec. 3.4) of max_new tokens after a HOST prompt of prompt_len >= 1 ids.
 * The prompt minus its last token is prefilled; every stage drafts at
 * most min(K_max, tokens still to emit - 1) tokens with skip_mask (HOST,
 * as in sd_forward), stopping right after a token whose top-1 probability
 * is below gamma (that token is still verified), then verifies them in one
 * forward of the full model and keeps the longest matching prefix plus the
 * model's next token.  The draft shares the KV cache: it reads the
 * committed positions and writes its own positions in the attention
 * sublayers it runs; verification overwrites them.  0 <= K_max <= 15.
 * out_tokens: HOST int32 [max_new].  stats may be NULL.  The host waits
 * for each draft step's exit decision through a pinned mailbox; no other
 * synchronisation happens per token.  Errors: INVALID_ARG, OOM, DEVICE. */
sd_status sd_self_spec_generate(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                const uint8_t *skip_mask, int32_t K_max, float gamma, int32_t *out_tokens,
                                sd_stats *stats);

/* sd_self_spec_generate with the adaptive threshold of Sec. 3.4 (Eqs. 2-4)
 * in place of a fixed gamma; params is a HOST sd_adaptive (no NaN fields).
 * The update runs on the device after each verification, with no extra
 * synchronisation.  Errors: INVALID_ARG, OOM, DEVICE. */
sd_status sd_self_spec_generate_adaptive(sd_model *model, const int32_t *prompt, int32_t prompt_len,
                                         int32_t max_new, const uint8_t *skip_mask, int32_t K_max,
                                         const sd_adaptive *params, int32_t *out_tokens, sd_stats *stats);

/* Greedy autoregressive decoding (Algorithm 1) with the same prefill
 * convention; one full-model forward per token, no per-token host sync. */
sd_status sd_autoregressive_generate(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                     int32_t *out_tokens, sd_stats *stats);

/* Sampling variant (the appendix's self-speculative decoding with random
 * sampling).  A row's distribution is warped: softmax(logits / temperature)
 * restricted to its top-p nucleus, the shortest run of tokens in
 * (probability descending, id ascending) order whose mass reaches top_p,
 * renormalised.  Every uniform is the top 24 bits of the first word of
 * Philox4x64-10 (Salmon et al., SC'11) with key (seed, 0) and counter
 * (output index, purpose, stage, 0); purposes: 0 draft draw, 1 acceptance
 * test, 2 the draw after the accepted drafts (and every autoregressive
 * draw, with stage = output index).  Identical inputs and seed give
 * identical tokens. */
typedef struct {
    float temperature; /* > 0, finite */
    float top_p;       /* in (0, 1] */
    uint64_t seed;
} sd_sampling;

/* Self-speculative sampling: drafts are drawn from the warped draft
 * distribution q, and a stage stops right after a draft whose warped
 * maximum is below the threshold (gamma, or the adaptive rule when adaptive
 * is not NULL, as in sd_self_spec_generate_adaptive).  Draft d at a
 * position is accepted when r < min(1, p(d) / q(d)), p the warped full-model
 * distribution there and r uniform; the first rejected position is redrawn
 * from max(0, p - q) normalised (from p if that is empty); a fully accepted
 * stage ends with a draw from p.  The emitted tokens are distributed as
 * autoregressive sampling from the full model.  Masses are exact sums of
 * 31-bit fixed-point weights.  Other arguments and errors as for
 * sd_self_spec_generate; sampling is a HOST sd_sampling; the vocabulary
 * must have at most 524288 ids (INVALID_ARG otherwise). */
sd_status sd_self_spec_sample(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                              const uint8_t *skip_mask, int32_t K_max, float gamma, const sd_adaptive *adaptive,
                              const sd_sampling *sampling, int32_t *out_tokens, sd_stats *stats);

/* Autoregressive sampling: token i is drawn from the warped full-model
 * distribution with the uniform of (i, purpose 2, stage i), so
 * sd_self_spec_sample with K_max = 0 returns the same tokens. */
sd_status sd_autoregressive_sample(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                   const sd_sampling *sampling, int32_t *out_tokens, sd_stats *stats);

/* Skip-set search (Sec. 3.3, Eq. 1): z* = argmin f(z) over sublayer masks
 * z in {0, 1}^L, by Bayesian optimisation for a fixed number of steps.
 * Host code; every evaluation of f is one call of the objective.
 *   - n_init initial masks, mask i with each bit set with probability
 *     0.6 i / n_init (mask 0 is empty);
 *   - surrogate: a zero-mean Gaussian process over the standardised
 *     observations (mean 0, population deviation 1; a deviation below 1e-12
 *     counts as 1), kernel exp(-hamming(a, b) / (length_scale L)), noise
 *     variance `noise` on the observations;
 *   - acquisition: expected improvement below the smallest standardised
 *     observation by xi, of the posterior of the noise-free value;
 *   - each step scores n_candidates masks, the first half 1 to 3 random
 *     flips of the incumbent (the best mask so far, first on ties), the
 *     rest random masks with one density drawn from [0, 0.6); masks
 *     evaluated before are dropped, the first maximiser of EI is evaluated,
 *     and a step with no new candidate evaluates nothing;
 *   - random numbers: top 24 bits of the first word of Philox4x64-10 with
 *     key (seed, 1), counter (index, purpose, sub-index, 0).
 * Limits: 1 <= L <= 1024, n_init + iterations <= 4096, n_candidates <= 65536. */
typedef enum { SD_SEARCH_MEASURED = 0, SD_SEARCH_MODELED = 1 } sd_search_objective;

typedef struct {
    int32_t n_init;       /* >= 1 */
    int32_t iterations;   /* BO steps after the initial masks, >= 0 */
    int32_t n_candidates; /* >= 1 */
    double length_scale;  /* > 0 */
    double noise;         /* > 0: observation noise variance of the standardised values */
    double xi;            /* finite */
    uint64_t seed;
    int32_t objective;    /* sd_search_skip_set only: an sd_search_objective */
    /* SD_SEARCH_MODELED costs (finite): a draft step costs cost[0] + cost[1] per
     * attention + cost[2] per MLP sublayer it runs; a verification cost[3]
     * + cost[4] per row (drafts + 1) */
    double cost[5];
} sd_search_params;

/* Outputs.  best_mask is required; the arrays may be NULL, else they hold
 * n_init + iterations entries of which the first n_evaluated are written. */
typedef struct {
    uint8_t *best_mask; /* HOST uint8 [L]: the evaluated mask of least f (the first on ties) */
    double best_value;
    int32_t n_evaluated;
    uint8_t *masks;     /* HOST uint8 [n_init + iterations][L]: evaluated masks in order */
    double *values;     /* HOST [n_init + iterations]: f of each */
    double *margins;    /* HOST [n_init + iterations]: EI of the chosen candidate minus the largest EI
                         * below it (infinity for the initial masks and for a single EI value) */
} sd_search_result;

/* The objective of sd_search_skip_set_fn: writes f(mask) to *value and
 * returns SD_OK, or another status, which stops the search with it. */
typedef sd_status (*sd_search_objective_fn)(const uint8_t *mask, int32_t n_dims, void *user, double *value);

/* Search over masks of n_dims bits with a caller's objective (finite values).
 * params->objective and cost are ignored.  Errors: INVALID_ARG (also for a
 * non-finite objective value or a surrogate that is not positive definite),
 * OOM, or the objective's status. */
sd_status sd_search_skip_set_fn(int32_t n_dims, const sd_search_params *params, sd_search_objective_fn objective,
                                void *user, sd_search_result *result);

/* Search of the model's skip mask (L = 2 n_layers, layout of sd_forward),
 * f(z) the time per emitted token of self-speculative decoding of max_new
 * tokens after each of n_prompts HOST prompts of prompt_len ids (row-major
 * [n_prompts][prompt_len]), with K_max and gamma (adaptive, when not NULL,
 * as in sd_self_spec_generate_adaptive).  SD_SEARCH_MEASURED: summed
 * decode_ms / (n_prompts max_new); SD_SEARCH_MODELED: the costs above summed
 * over the stages of every decode / (n_prompts max_new), a function of the
 * decoded tokens only.  Errors: as sd_self_spec_generate and
 * sd_search_skip_set_fn. */
sd_status sd_search_skip_set(sd_model *model, const int32_t *prompts, int32_t n_prompts, int32_t prompt_len,
                             int32_t max_new, int32_t K_max, float gamma, const sd_adaptive *adaptive,
                             const sd_search_params *params, sd_search_result *result);

/* Measurement hook.  Selects one linear-layer class whose launches the
 * library brackets with HIP events on its stream: layer 0 = QKV, 1 = attention
 * output, 2 = gate/up, 3 = down, 4 = lm-head; rows = 1, 2 or 16 selects the
 * kernel family used for forwards of one row, up to two rows, or more rows.
 * layer = -1 turns timing off.  The launches of the class in one of every
 * 16 forwards of that row regime are timed, with start/stop events the
 * runtime attaches to the dispatch itself (the kernel's own start and end);
 * at most 65536 launches per call are timed.  Resets the totals and the
 * forward count.  Errors: INVALID_ARG. */
sd_status sd_model_time_kernel(sd_model *model, int32_t layer, int32_t rows);

/* Totals of the timed class since sd_model_time_kernel: launches, summed
 * GPU milliseconds, the kernel symbol as a profiler prints it (written to
 * kernel_name, NUL-terminated, truncated to name_cap), and the weight
 * matrix shape n x k of one launch.  Any output pointer may be NULL. */
sd_status sd_model_kernel_time(sd_model *model, int64_t *launches, double *total_ms, char *kernel_name,
                               int32_t name_cap, int64_t *n, int64_t *k);

/* Message of the last non-OK status returned to this thread ("" if none). */
/* Measurement (the achievable ceiling beside the 8 TB/s peak): decoding is
 * bound by memory bandwidth (Sec. 1, 3.1), so the GB/s of the decoding
 * kernels are also read against what a plain streaming read reaches on this
 * GPU.  Reads `bytes` (a positive multiple of 16) of the DEVICE buffer buf
 * (16-byte aligned) `iters` times with 16-byte non-temporal loads, the
 * pattern of the weight-streaming layers, loads_in_flight (2, 4, 8 or 16)
 * per thread, on wg_per_cu x (compute units) work-groups of 256 threads on
 * hip_stream (NULL: the null stream).  *ms_out
 * receives the mean duration of one read, from events attached to each
 * dispatch.  sink is a DEVICE buffer of at least 4 bytes that the probe may
 * write (it keeps the loads from being optimised away).  Errors:
 * INVALID_ARG, DEVICE. */
sd_status sd_measure_read_bandwidth(const void *buf, size_t bytes, int32_t wg_per_cu, int32_t loads_in_flight,
                                    int32_t iters, void *sink, void *hip_stream, double *ms_out);

const char *sd_last_error(void);

/* Library version string. */
const char *sd_version(void);

#ifdef __cplusplus
}
#endif

#endif
