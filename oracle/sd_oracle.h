/* Plain CPU oracle for greedy self-speculative decoding (Draft & Verify,
 * Zhang et al., arXiv 2309.08168).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes,
 * links or calls this code; only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark use it.  It shares no code, header,
 * table or helper with the GPU path.
 *
 * Arithmetic is float64 throughout.  Weights are read as stored (float32,
 * or bfloat16 bit patterns expanded exactly).  The KV cache holds each
 * element in the model's storage precision: exact for float32 models,
 * rounded to the nearest bfloat16 for bfloat16 models (the precision the
 * paper's models run in).
 * Every output element is a sequential reduction over its inputs in index
 * order, so a row's result does not depend on how many rows share the call
 * or on the thread count.  Argmax and the top-1 probability are decided on
 * logits rounded to float32, the precision the GPU path takes those
 * decisions in.
 *
 * Model (pre-norm LLaMA decoder, the models the paper evaluates, Sec. 4.1):
 *   h = E[x];  per layer l: attention sublayer unless skip[2l], MLP sublayer
 *   unless skip[2l+1];  logits = W_lm * RMSNorm(h).
 * A skipped sublayer is the identity on the residual stream (Sec. 3.2: the
 * draft model bypasses intermediate layers); it computes nothing and writes
 * no KV.
 */
#ifndef SD_ORACLE_H
#define SD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
    double rms_eps, rope_base;
    int32_t wdtype; /* 0: float32 weights, 1: bfloat16 bit patterns (uint16) */
} orc_config;

/* Host pointers, row-major [out, in].  w_qkv = [(H + 2 KVH) dh, d] with q
 * rows, then k rows, then v rows; w_gate_up = [2F, d], gate rows then up
 * rows.  Per-layer members point to arrays of n_layers pointers, copied at
 * create time; the tensors themselves are borrowed and must outlive the
 * model. */
typedef struct {
    const void *tok_emb, *final_norm, *lm_head;
    const void *const *attn_norm, *const *w_qkv, *const *w_o;
    const void *const *mlp_norm, *const *w_gate_up, *const *w_down;
} orc_weights;

typedef struct orc_model orc_model;
typedef struct orc_cache orc_cache;

typedef struct {
    int64_t n_stages;      /* drafting/verification stages */
    int64_t n_drafted;     /* sum over stages of drafted tokens k_e */
    int64_t n_accepted;    /* sum over stages of accepted drafts n_e */
    int64_t n_emitted;     /* tokens emitted (= max_new) */
    int64_t n_draft_steps; /* draft forwards run (= n_drafted) */
    double min_gamma_gap;  /* min over draft steps of |p_max - gamma| */
    double min_draft_margin; /* min over greedy draft steps of the top-2 logit margin (inf when sampling) */
} orc_sd_stats;

/* Errors: 0 ok, -1 invalid argument, -2 KV capacity exceeded, -3 out of memory. */

orc_model *orc_create(const orc_config *cfg, const orc_weights *w);
void orc_destroy(orc_model *m);
int32_t orc_num_threads(void);

orc_cache *orc_cache_create(const orc_model *m, int32_t capacity);
void orc_cache_destroy(orc_cache *c);
int32_t orc_cache_length(const orc_cache *c);
int orc_cache_truncate(orc_cache *c, int32_t len);
/* Load externally generated K/V for positions [0, len): kv is laid out
 * [n_layers][2 (K, V)][n_kv_heads][len][head_dim] in kv_dtype (0 float32,
 * 1 bfloat16 bits); sets the cache length to len. */
int orc_cache_load(orc_cache *c, const void *kv, int32_t len, int32_t kv_dtype);

/* One forward of n rows at positions [len, len + n) of the cache; writes
 * K/V of every non-skipped attention sublayer and sets len += n.  skip is
 * uint8[2 * n_layers] or NULL (full model).  Outputs are optional:
 * logits float64 [n][vocab]; argmax int32 [n] (lowest id among equal float32
 * logits); pmax float32 [n] = 1 / sum_v exp(l_v - l_max) over float32
 * logits; margin float64 [n] = top-1 minus top-2 float64 logit. */
int orc_forward(orc_model *m, orc_cache *c, const int32_t *tokens, int32_t n, const uint8_t *skip,
                double *logits, int32_t *argmax, float *pmax, double *margin);

/* Greedy autoregressive decoding (Alg. 1).  out int32 [max_new]; margin
 * float64 [max_new] optional: top-2 margin of the logits each token came
 * from. */
int orc_generate_ar(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                    int32_t *out, double *margin);

/* Greedy self-speculative decoding (Alg. 2 with the static-threshold draft
 * exit of Sec. 3.4).  stage_log int32 [max_new][2] optional: (k_e, n_e) per
 * stage; draft_pmax float32 [max_new * K_max] optional: p_max of every
 * draft step in order; margin as for orc_generate_ar (from the
 * verification forward). */
int orc_generate_sd(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                    const uint8_t *skip, int32_t k_max, float gamma, int32_t *out, double *margin,
                    orc_sd_stats *stats, int32_t *stage_log, float *draft_pmax);

/* Adaptive draft exit (Sec. 3.4, Eqs. 2-4), updated after every
 * verification stage. */
typedef struct {
    double gamma0;  /* initial threshold */
    double alpha;   /* target acceptance rate */
    double epsilon; /* step of the threshold update */
    double beta1;   /* smoothing of the acceptance rate */
    double beta2;   /* smoothing of the threshold */
} orc_adaptive;

/* Greedy self-speculative decoding with the adaptive threshold; arguments as
 * for orc_generate_sd.  gamma_log float32 [max_new] optional: the threshold
 * each stage drafted with. */
int orc_generate_sd_adaptive(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                             const uint8_t *skip, int32_t k_max, const orc_adaptive *ad, int32_t *out,
                             double *margin, orc_sd_stats *stats, int32_t *stage_log, float *draft_pmax,
                             float *gamma_log);

/* ------------------------------------------------------------------------
 * Sampling variant (appendix, the sampling form of self-speculative
 * decoding): tokens are drawn from the temperature- and top-p-warped
 * distributions of the draft (q) and full (p) models; a draft d is accepted
 * when r < min(1, p(d) / q(d)) for a uniform r, the first rejected position
 * is redrawn from max(0, p - q) normalised, and a fully accepted stage ends
 * with a draw from p.  Every uniform comes from Philox4x64-10 keyed by the
 * seed, with the counter (output index, purpose, stage, 0).
 */
typedef struct {
    double temperature; /* > 0 */
    double top_p;       /* in (0, 1] */
    uint64_t seed;
} orc_sampling;

enum { ORC_U_DRAFT = 0, ORC_U_ACCEPT = 1, ORC_U_FINAL = 2 };

/* Philox4x64-10 (Salmon et al., SC'11): out = the 4 words of block ctr under key. */
void orc_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
/* The uniform of (index, purpose, stage): (word 0 >> 40) * 2^-24, in [0, 1). */
double orc_uniform(uint64_t seed, int64_t index, int32_t purpose, int64_t stage);

/* The warped distribution of one row of logits (decided on their float32
 * roundings): softmax(l / T), restricted to the shortest prefix of tokens in
 * (probability descending, id ascending) order whose mass reaches top_p,
 * renormalised.  pi float64 [V]; returns the kept count.  cut_margin
 * (optional): distance, in probability, of top_p from the masses just
 * without and with the last kept token (infinity when top_p >= 1). */
int32_t orc_warp(const double *logits, int32_t V, double temperature, double top_p, double *pi,
                 double *cut_margin);

/* Self-speculative sampling.  ad == NULL: static threshold gamma; otherwise
 * the adaptive rule.  margin float64 [max_new] (optional): for each emitted
 * token the smallest margin of the decisions that produced it (the draw's
 * distance to its CDF boundaries, the acceptance test's |r - min(1, p/q)|,
 * the top-p cut margins of the rows involved).  draft_qmax float32
 * [max_new * K_max] (optional): the warped draft maximum of each draft
 * step.  Other outputs as for orc_generate_sd_adaptive. */
int orc_generate_sd_sample(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                           const uint8_t *skip, int32_t k_max, float gamma, const orc_adaptive *ad,
                           const orc_sampling *sp, int32_t *out, double *margin, orc_sd_stats *stats,
                           int32_t *stage_log, float *draft_qmax, float *gamma_log);

/* Autoregressive sampling: token i is drawn from the warped full-model
 * distribution with the uniform of (i, ORC_U_FINAL, i). */
int orc_generate_ar_sample(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                           const orc_sampling *sp, int32_t *out, double *margin);

/* ------------------------------------------------------------------------
 * FP8 draft weights (the adaptation appendix combines self-speculative
 * decoding with FP8 and FP4 weights; here only a copy of the draft's
 * weights is quantized, and verification keeps the stored bf16 weights).
 * OCP FP8 E4M3 with one power-of-two scale 2^e per output row, e the
 * smallest integer with max|W[n][:]| * 2^-e <= 448; the byte is the nearest
 * E4M3 value (ties to even) of W[n][k] * 2^-e.
 */

/* The value of an E4M3 byte (NaN for S.1111.111). */
double orc_fp8_value(uint8_t b);

/* Quantizes a bf16 matrix [n_rows][n_cols]: bytes q [n_rows][n_cols],
 * exponents e [n_rows]. */
int orc_quantize_fp8_rows(const uint16_t *w, int64_t n_rows, int64_t n_cols, uint8_t *q, int32_t *e);

/* bf16 models: quantizes the QKV, output, gate/up and down weights of the
 * sublayers skip keeps (0 entries); from then on every forward with a skip
 * mask (a draft forward) reads those copies, and the full model the stored
 * weights.  skip == NULL removes them.  Errors: -1 argument, -3 memory. */
int orc_set_draft_fp8(orc_model *m, const uint8_t *skip);

#ifdef __cplusplus
}
#endif

#endif
