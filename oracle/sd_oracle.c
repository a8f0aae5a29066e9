/* Plain CPU oracle for greedy self-speculative decoding.  TEST INFRASTRUCTURE
 * ONLY; see sd_oracle.h for what it computes and who may use it.
 *
 * Sections of the paper (arXiv 2309.08168) followed here:
 *   - greedy autoregressive decoding: Sec. 3.1, Algorithm 1;
 *   - self-speculative decoding: Sec. 3.2, Algorithm 2 (draft with the
 *     skipped sublayers, verify all drafts in one forward of the original
 *     model, keep the longest matching prefix, replace the first mismatch or
 *     add one bonus token when all drafts match);
 *   - draft exit: Sec. 3.4 and Algorithm 3 (stop drafting right after a
 *     draft token whose top-1 probability is below gamma);
 *   - skipping granularity: Sec. 3.3 and the skip-pattern figure (z has one
 *     entry per attention and per MLP sublayer).
 * Readings where the paper is silent are marked "Reading:" below.
 */
#include "sd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

enum { FP8_QKV = 0, FP8_O = 1, FP8_GATE_UP = 2, FP8_DOWN = 3, FP8_KINDS = 4 };

struct orc_model {
    orc_config c;
    const void *tok_emb, *final_norm, *lm_head;
    const void **attn_norm, **w_qkv, **w_o, **mlp_norm, **w_gate_up, **w_down;
    /* FP8 draft copies (orc_set_draft_fp8): per kind and layer, the E4M3
     * bytes [N][K] and the per-row scale exponents [N], or NULL */
    uint8_t **fp8_q[FP8_KINDS];
    int32_t **fp8_e[FP8_KINDS];
};

struct orc_cache {
    const orc_model *m;
    int32_t cap, len;
    double *kv; /* [n_layers][2][n_kv_heads][cap][head_dim] */
};

/* ------------------------------------------------------------------------ */
/* weights */

static double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double wval(const orc_model *m, const void *p, int64_t i)
{
    if (m->c.wdtype == 1)
        return bf16_to_double(((const uint16_t *)p)[i]);
    return (double)((const float *)p)[i];
}

static void wrow(const orc_model *m, const void *p, int64_t row, int64_t ncols, double *dst)
{
    for (int64_t k = 0; k < ncols; ++k)
        dst[k] = wval(m, p, row * ncols + k);
}

/* Reading: the models the paper evaluates run in bfloat16 (its adaptation
 * appendix names bf16 the default), so their KV caches hold bfloat16
 * values.  For bf16 models the cache stores each K/V element rounded to the
 * nearest bfloat16 (ties to even); float32 models keep it exact. */
static double kv_store_value(const orc_model *m, double x)
{
    if (m->c.wdtype != 1 || x == 0.0 || !isfinite(x))
        return x;
    int e;
    const double f = frexp(x, &e);       /* x = f * 2^e, 0.5 <= |f| < 1 */
    return ldexp(rint(ldexp(f, 8)), e - 8); /* 8 significant bits, ties to even */
}

static const void **copy_ptrs(const void *const *src, int n)
{
    const void **dst = (const void **)malloc(sizeof(void *) * (size_t)n);
    if (dst)
        memcpy(dst, src, sizeof(void *) * (size_t)n);
    return dst;
}

orc_model *orc_create(const orc_config *cfg, const orc_weights *w)
{
    if (!cfg || !w || cfg->n_layers < 1 || cfg->d_model < 1 || cfg->n_heads < 1 || cfg->n_kv_heads < 1 ||
        cfg->head_dim < 2 || (cfg->head_dim & 1) || cfg->n_heads % cfg->n_kv_heads || cfg->ffn_dim < 1 ||
        cfg->vocab < 2 || (cfg->wdtype != 0 && cfg->wdtype != 1))
        return NULL;
    orc_model *m = (orc_model *)calloc(1, sizeof *m);
    if (!m)
        return NULL;
    m->c = *cfg;
    m->tok_emb = w->tok_emb;
    m->final_norm = w->final_norm;
    m->lm_head = w->lm_head;
    int L = cfg->n_layers;
    m->attn_norm = copy_ptrs(w->attn_norm, L);
    m->w_qkv = copy_ptrs(w->w_qkv, L);
    m->w_o = copy_ptrs(w->w_o, L);
    m->mlp_norm = copy_ptrs(w->mlp_norm, L);
    m->w_gate_up = copy_ptrs(w->w_gate_up, L);
    m->w_down = copy_ptrs(w->w_down, L);
    if (!m->attn_norm || !m->w_qkv || !m->w_o || !m->mlp_norm || !m->w_gate_up || !m->w_down) {
        orc_destroy(m);
        return NULL;
    }
    return m;
}

static void free_draft_fp8(orc_model *m);

void orc_destroy(orc_model *m)
{
    if (!m)
        return;
    free_draft_fp8(m);
    free((void *)m->attn_norm);
    free((void *)m->w_qkv);
    free((void *)m->w_o);
    free((void *)m->mlp_norm);
    free((void *)m->w_gate_up);
    free((void *)m->w_down);
    free(m);
}

int32_t orc_num_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* KV cache */

static size_t kv_index(const orc_cache *c, int l, int kv, int g, int pos)
{
    const orc_config *cf = &c->m->c;
    return ((((size_t)l * 2 + (size_t)kv) * (size_t)cf->n_kv_heads + (size_t)g) * (size_t)c->cap + (size_t)pos) *
           (size_t)cf->head_dim;
}

orc_cache *orc_cache_create(const orc_model *m, int32_t capacity)
{
    if (!m || capacity < 1)
        return NULL;
    orc_cache *c = (orc_cache *)calloc(1, sizeof *c);
    if (!c)
        return NULL;
    c->m = m;
    c->cap = capacity;
    size_t n = (size_t)m->c.n_layers * 2 * (size_t)m->c.n_kv_heads * (size_t)capacity * (size_t)m->c.head_dim;
    c->kv = (double *)calloc(n, sizeof(double));
    if (!c->kv) {
        free(c);
        return NULL;
    }
    return c;
}

void orc_cache_destroy(orc_cache *c)
{
    if (!c)
        return;
    free(c->kv);
    free(c);
}

int32_t orc_cache_length(const orc_cache *c) { return c ? c->len : -1; }

int orc_cache_truncate(orc_cache *c, int32_t len)
{
    if (!c || len < 0 || len > c->len)
        return -1;
    c->len = len;
    return 0;
}

int orc_cache_load(orc_cache *c, const void *kv, int32_t len, int32_t kv_dtype)
{
    if (!c || !kv || len < 0 || (kv_dtype != 0 && kv_dtype != 1))
        return -1;
    if (len > c->cap)
        return -2;
    const orc_config *cf = &c->m->c;
    size_t src = 0;
    for (int l = 0; l < cf->n_layers; ++l)
        for (int kvi = 0; kvi < 2; ++kvi)
            for (int g = 0; g < cf->n_kv_heads; ++g)
                for (int p = 0; p < len; ++p) {
                    double *dst = c->kv + kv_index(c, l, kvi, g, p);
                    for (int e = 0; e < cf->head_dim; ++e, ++src)
                        dst[e] = kv_dtype == 1 ? bf16_to_double(((const uint16_t *)kv)[src])
                                               : (double)((const float *)kv)[src];
                }
    c->len = len;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* building blocks of the LLaMA decoder */

/* y[r][n] = sum_k W[n][k] x[r][k]; W row-major [N][K].  Each output is a
 * sequential sum over k, so it does not depend on nr or on threads. */
static void linear(const orc_model *m, const void *W, int64_t N, int64_t K, const double *x, int nr, double *y)
{
#pragma omp parallel
    {
        double *row = (double *)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            wrow(m, W, n, K, row);
            for (int r = 0; r < nr; ++r) {
                const double *xr = x + (int64_t)r * K;
                double acc = 0.0;
                for (int64_t k = 0; k < K; ++k)
                    acc += row[k] * xr[k];
                y[(int64_t)r * N + n] = acc;
            }
        }
        free(row);
    }
}

/* The same with FP8 draft weights: W[n][k] = value(q[n][k]) * 2^e[n], every
 * output again a sequential sum over k. */
static void linear_fp8(const uint8_t *q, const int32_t *e, int64_t N, int64_t K, const double *x, int nr, double *y)
{
#pragma omp parallel
    {
        double *row = (double *)malloc(sizeof(double) * (size_t)K);
#pragma omp for schedule(static)
        for (int64_t n = 0; n < N; ++n) {
            for (int64_t k = 0; k < K; ++k)
                row[k] = ldexp(orc_fp8_value(q[n * K + k]), e[n]);
            for (int r = 0; r < nr; ++r) {
                const double *xr = x + (int64_t)r * K;
                double acc = 0.0;
                for (int64_t k = 0; k < K; ++k)
                    acc += row[k] * xr[k];
                y[(int64_t)r * N + n] = acc;
            }
        }
        free(row);
    }
}

/* A linear layer of a draft forward (skip mask given) reads the FP8 copy
 * when the model has one for (kind, layer); every other forward reads the
 * stored weights. */
static void linear_layer(const orc_model *m, int kind, int l, const uint8_t *skip, const void *W, int64_t N,
                         int64_t K, const double *x, int nr, double *y)
{
    if (skip && m->fp8_q[kind] && m->fp8_q[kind][l])
        linear_fp8(m->fp8_q[kind][l], m->fp8_e[kind][l], N, K, x, nr, y);
    else
        linear(m, W, N, K, x, nr, y);
}

/* RMSNorm: u = g * h / sqrt(mean(h^2) + eps). */
static void rmsnorm(const orc_model *m, const void *g, const double *h, double *u)
{
    int d = m->c.d_model;
    double ss = 0.0;
    for (int k = 0; k < d; ++k)
        ss += h[k] * h[k];
    double inv = 1.0 / sqrt(ss / (double)d + m->c.rms_eps);
    for (int k = 0; k < d; ++k)
        u[k] = wval(m, g, k) * (h[k] * inv);
}

/* Reading: rotary position embedding in the rotate-half form of the LLaMA-2
 * models the paper evaluates: element i pairs with i + dh/2, angle
 * pos * base^(-2i/dh). */
static void rope(const orc_model *m, double *x, int n_heads, int pos)
{
    int dh = m->c.head_dim, half = dh / 2;
    for (int h = 0; h < n_heads; ++h) {
        double *v = x + (int64_t)h * dh;
        for (int i = 0; i < half; ++i) {
            double theta = pow(m->c.rope_base, -2.0 * (double)i / (double)dh);
            double ang = (double)pos * theta;
            double cs = cos(ang), sn = sin(ang);
            double a = v[i], b = v[i + half];
            v[i] = a * cs - b * sn;
            v[i + half] = b * cs + a * sn;
        }
    }
}

static double silu(double a) { return a / (1.0 + exp(-a)); }

/* Causal attention of one query row at position pos over cached keys
 * [0, pos] of layer l; grouped-query heads share KV head j / (H / KVH). */
static void attend(const orc_cache *c, int l, const double *q, int pos, double *o, double *scores)
{
    const orc_config *cf = &c->m->c;
    int H = cf->n_heads, dh = cf->head_dim, grp = cf->n_heads / cf->n_kv_heads;
    double scale = 1.0 / sqrt((double)dh);
    for (int j = 0; j < H; ++j) {
        int g = j / grp;
        const double *qj = q + (int64_t)j * dh;
        double mx = -INFINITY;
        for (int i = 0; i <= pos; ++i) {
            const double *ki = c->kv + kv_index(c, l, 0, g, i);
            double s = 0.0;
            for (int e = 0; e < dh; ++e)
                s += qj[e] * ki[e];
            scores[i] = s * scale;
            if (scores[i] > mx)
                mx = scores[i];
        }
        double den = 0.0;
        for (int i = 0; i <= pos; ++i) {
            scores[i] = exp(scores[i] - mx);
            den += scores[i];
        }
        double *oj = o + (int64_t)j * dh;
        for (int e = 0; e < dh; ++e)
            oj[e] = 0.0;
        for (int i = 0; i <= pos; ++i) {
            const double *vi = c->kv + kv_index(c, l, 1, g, i);
            double a = scores[i] / den;
            for (int e = 0; e < dh; ++e)
                oj[e] += a * vi[e];
        }
    }
}

/* Greedy head of one row: argmax (lowest id among equal float32 logits),
 * top-1 probability from the float32 logits, top-2 margin of the float64
 * logits. */
static void greedy_head(const double *logit, int V, int32_t *amax, float *pmax, double *margin)
{
    int best = 0;
    float bestf = (float)logit[0];
    for (int v = 1; v < V; ++v) {
        float f = (float)logit[v];
        if (f > bestf) {
            bestf = f;
            best = v;
        }
    }
    double den = 0.0;
    for (int v = 0; v < V; ++v)
        den += exp((double)(float)logit[v] - (double)bestf);
    double t1 = -INFINITY, t2 = -INFINITY;
    for (int v = 0; v < V; ++v) {
        if (logit[v] > t1) {
            t2 = t1;
            t1 = logit[v];
        } else if (logit[v] > t2) {
            t2 = logit[v];
        }
    }
    if (amax)
        *amax = best;
    if (pmax)
        *pmax = (float)(1.0 / den);
    if (margin)
        *margin = t1 - t2;
}

/* ------------------------------------------------------------------------ */
/* forward */

int orc_forward(orc_model *m, orc_cache *c, const int32_t *tokens, int32_t n, const uint8_t *skip, double *logits,
                int32_t *argmax, float *pmax, double *margin)
{
    if (!m || !c || c->m != m || !tokens || n < 1)
        return -1;
    const orc_config *cf = &m->c;
    for (int r = 0; r < n; ++r)
        if (tokens[r] < 0 || tokens[r] >= cf->vocab)
            return -1;
    if (skip)
        for (int i = 0; i < 2 * cf->n_layers; ++i)
            if (skip[i] > 1)
                return -1;
    if ((int64_t)c->len + n > c->cap)
        return -2;

    const int d = cf->d_model, H = cf->n_heads, KVH = cf->n_kv_heads, dh = cf->head_dim, F = cf->ffn_dim;
    const int V = cf->vocab, nqkv = (H + 2 * KVH) * dh, start = c->len;
    double *h = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *u = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *t = (double *)malloc(sizeof(double) * (size_t)n * d);
    double *qkv = (double *)malloc(sizeof(double) * (size_t)n * nqkv);
    double *o = (double *)malloc(sizeof(double) * (size_t)n * H * dh);
    double *gu = (double *)malloc(sizeof(double) * (size_t)n * 2 * F);
    double *mm = (double *)malloc(sizeof(double) * (size_t)n * F);
    int rc = 0;
    if (!h || !u || !t || !qkv || !o || !gu || !mm) {
        rc = -3;
        goto done;
    }

    for (int r = 0; r < n; ++r)
        wrow(m, m->tok_emb, tokens[r], d, h + (int64_t)r * d);

    for (int l = 0; l < cf->n_layers; ++l) {
        if (!(skip && skip[2 * l])) {
            for (int r = 0; r < n; ++r)
                rmsnorm(m, m->attn_norm[l], h + (int64_t)r * d, u + (int64_t)r * d);
            linear_layer(m, FP8_QKV, l, skip, m->w_qkv[l], nqkv, d, u, n, qkv);
            /* all rows of the block write their K/V first, then attend */
            for (int r = 0; r < n; ++r) {
                double *row = qkv + (int64_t)r * nqkv;
                rope(m, row, H, start + r);
                rope(m, row + (int64_t)H * dh, KVH, start + r);
                for (int g = 0; g < KVH; ++g) {
                    double *kd = c->kv + kv_index(c, l, 0, g, start + r);
                    double *vd = c->kv + kv_index(c, l, 1, g, start + r);
                    for (int e = 0; e < dh; ++e) {
                        kd[e] = kv_store_value(m, row[(int64_t)(H + g) * dh + e]);
                        vd[e] = kv_store_value(m, row[(int64_t)(H + KVH + g) * dh + e]);
                    }
                }
            }
#pragma omp parallel
            {
                double *scores = (double *)malloc(sizeof(double) * (size_t)(start + n));
#pragma omp for schedule(static)
                for (int r = 0; r < n; ++r)
                    attend(c, l, qkv + (int64_t)r * nqkv, start + r, o + (int64_t)r * H * dh, scores);
                free(scores);
            }
            linear_layer(m, FP8_O, l, skip, m->w_o[l], d, (int64_t)H * dh, o, n, t);
            for (int64_t i = 0; i < (int64_t)n * d; ++i)
                h[i] += t[i];
        }
        if (!(skip && skip[2 * l + 1])) {
            for (int r = 0; r < n; ++r)
                rmsnorm(m, m->mlp_norm[l], h + (int64_t)r * d, u + (int64_t)r * d);
            linear_layer(m, FP8_GATE_UP, l, skip, m->w_gate_up[l], 2 * (int64_t)F, d, u, n, gu);
            for (int r = 0; r < n; ++r)
                for (int f = 0; f < F; ++f) {
                    const double *gr = gu + (int64_t)r * 2 * F;
                    mm[(int64_t)r * F + f] = silu(gr[f]) * gr[F + f];
                }
            linear_layer(m, FP8_DOWN, l, skip, m->w_down[l], d, F, mm, n, t);
            for (int64_t i = 0; i < (int64_t)n * d; ++i)
                h[i] += t[i];
        }
    }
    c->len = start + n;

    if (logits || argmax || pmax || margin) {
        double *lg = logits ? logits : (double *)malloc(sizeof(double) * (size_t)n * V);
        if (!lg) {
            rc = -3;
            goto done;
        }
        for (int r = 0; r < n; ++r)
            rmsnorm(m, m->final_norm, h + (int64_t)r * d, u + (int64_t)r * d);
        linear(m, m->lm_head, V, d, u, n, lg);
        for (int r = 0; r < n; ++r)
            greedy_head(lg + (int64_t)r * V, V, argmax ? argmax + r : NULL, pmax ? pmax + r : NULL,
                        margin ? margin + r : NULL);
        if (!logits)
            free(lg);
    }
done:
    free(h);
    free(u);
    free(t);
    free(qkv);
    free(o);
    free(gu);
    free(mm);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* decoding */

/* Reading: the prompt minus its last token fills the cache; the last prompt
 * token is the first input of decoding.  The same invariant holds after
 * every step of both decoders: the cache holds every committed token but
 * the last one. */
static int prefill(orc_model *m, orc_cache *c, const int32_t *prompt, int32_t t)
{
    if (t > 1)
        return orc_forward(m, c, prompt, t - 1, NULL, NULL, NULL, NULL, NULL);
    return 0;
}

static int check_prompt(const orc_model *m, const int32_t *prompt, int32_t t)
{
    if (!prompt || t < 1)
        return -1;
    for (int i = 0; i < t; ++i)
        if (prompt[i] < 0 || prompt[i] >= m->c.vocab)
            return -1;
    return 0;
}

int orc_generate_ar(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new, int32_t *out, double *margin)
{
    if (!m || max_new < 0 || (max_new > 0 && !out) || check_prompt(m, prompt, t))
        return -1;
    orc_cache *c = orc_cache_create(m, t + max_new + 1);
    if (!c)
        return -3;
    int rc = prefill(m, c, prompt, t);
    int32_t last = prompt[t - 1];
    /* Algorithm 1: x_{i+1} = argmax p(x | x_1..x_i), one token per forward. */
    for (int i = 0; rc == 0 && i < max_new; ++i) {
        int32_t y;
        rc = orc_forward(m, c, &last, 1, NULL, NULL, &y, NULL, margin ? margin + i : NULL);
        out[i] = y;
        last = y;
    }
    orc_cache_destroy(c);
    return rc;
}

/* Reading: at most K drafts per stage, and never more than the tokens still
 * to emit minus the one the verification adds. */
static int32_t stage_budget(int32_t k_max, int32_t max_new, int32_t emitted)
{
    int32_t kcap = k_max;
    if (kcap > max_new - emitted - 1)
        kcap = max_new - emitted - 1;
    return kcap;
}

/* Adaptive threshold, after the verification stage (Eqs. 2-4): the stage's
 * acceptance rate AR_e = n_e / k_e is smoothed into AR (AR = AR_e at the
 * first stage), the threshold moves by epsilon up when AR is at most the
 * target alpha and down otherwise, and the move is smoothed by beta2.
 * Reading: a stage without drafts (k_e = 0, only at the end of generation or
 * with K = 0) says nothing about acceptance and leaves AR and gamma as they
 * are.  Returns the threshold of the next stage. */
typedef struct {
    double ar, gamma_d; /* gamma_d: the threshold in float64; the exit test uses it rounded to float32 */
    int64_t n_updates;
} adapt_state;

static float adapt_threshold(const orc_adaptive *ad, int32_t k, int32_t na, adapt_state *s, float gamma)
{
    if (!ad || k <= 0)
        return gamma;
    double ar = s->ar, gamma_d = s->gamma_d;
    const int64_t n_updates = s->n_updates;
    const double ar_e = (double)na / (double)k;
    ar = n_updates == 0 ? ar_e : ad->beta1 * ar + (1.0 - ad->beta1) * ar_e;
    const double gamma_t = ar <= ad->alpha ? gamma_d + ad->epsilon : gamma_d - ad->epsilon;
    gamma_d = ad->beta2 * gamma_d + (1.0 - ad->beta2) * gamma_t;
    s->ar = ar;
    s->gamma_d = gamma_d;
    s->n_updates = n_updates + 1;
    return (float)gamma_d;
}

/* Self-speculative decoding; ad == NULL keeps the threshold fixed at gamma,
 * otherwise it starts at ad->gamma0 and follows Eqs. 2-4. */
static int generate_sd(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new, const uint8_t *skip,
                       int32_t k_max, float gamma, const orc_adaptive *ad, int32_t *out, double *margin,
                       orc_sd_stats *stats, int32_t *stage_log, float *draft_pmax, float *gamma_log)
{
    if (!m || max_new < 0 || (max_new > 0 && !out) || k_max < 0 || gamma != gamma || check_prompt(m, prompt, t))
        return -1;
    adapt_state as = {0.0, ad ? ad->gamma0 : (double)gamma, 0};
    if (ad)
        gamma = (float)as.gamma_d;
    if (skip)
        for (int i = 0; i < 2 * m->c.n_layers; ++i)
            if (skip[i] > 1)
                return -1;
    orc_sd_stats st;
    memset(&st, 0, sizeof st);
    st.min_gamma_gap = INFINITY;
    st.min_draft_margin = INFINITY;
    /* Reading: the draft shares the one KV cache.  Draft steps write K/V of
     * the non-skipped attention sublayers at the draft positions; the
     * verification forward overwrites those positions at every layer, and
     * acceptance rolls the length back to the committed tokens. */
    orc_cache *c = orc_cache_create(m, t + max_new + k_max + 1);
    int32_t *draft = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k_max + 1));
    int32_t *rows = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k_max + 1));
    int32_t *y = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k_max + 1));
    double *ymargin = (double *)malloc(sizeof(double) * (size_t)(k_max + 1));
    if (!c || !draft || !rows || !y || !ymargin) {
        orc_cache_destroy(c);
        free(draft);
        free(rows);
        free(y);
        free(ymargin);
        return -3;
    }
    int rc = prefill(m, c, prompt, t);
    int32_t last = prompt[t - 1];
    int32_t emitted = 0;

    while (rc == 0 && emitted < max_new) {
        const int32_t lc = c->len; /* committed length: the cache holds all but `last` */
        const int32_t kcap = stage_budget(k_max, max_new, emitted);

        /* Drafting stage: greedy tokens of the model with the skip set
         * bypassed; exit right after a token whose top-1 probability is
         * below gamma (that token is still verified). */
        int32_t k = 0;
        for (int32_t j = 0; j < kcap; ++j) {
            int32_t in = j == 0 ? last : draft[j - 1];
            float p;
            double dm;
            rc = orc_forward(m, c, &in, 1, skip, NULL, &draft[j], &p, &dm);
            if (rc)
                break;
            if (dm < st.min_draft_margin)
                st.min_draft_margin = dm;
            if (draft_pmax)
                draft_pmax[st.n_draft_steps] = p;
            st.n_draft_steps++;
            double gap = fabs((double)p - (double)gamma);
            if (gap < st.min_gamma_gap)
                st.min_gamma_gap = gap;
            k = j + 1;
            if (p < gamma)
                break;
        }
        if (rc)
            break;

        /* Verification stage: one forward of the original model over the
         * last committed token and all drafts, at positions lc .. lc + k. */
        rc = orc_cache_truncate(c, lc);
        if (rc)
            break;
        rows[0] = last;
        for (int32_t j = 0; j < k; ++j)
            rows[j + 1] = draft[j];
        rc = orc_forward(m, c, rows, k + 1, NULL, NULL, y, NULL, ymargin);
        if (rc)
            break;

        /* Accept the longest prefix of drafts that the original model would
         * have produced; the model's own token follows it (the correction
         * at the first mismatch, or the bonus token when all match). */
        int32_t na = 0;
        while (na < k && draft[na] == y[na])
            ++na;
        for (int32_t j = 0; j < na; ++j) {
            if (margin)
                margin[emitted] = ymargin[j];
            out[emitted++] = draft[j];
        }
        if (margin)
            margin[emitted] = ymargin[na];
        out[emitted++] = y[na];
        last = y[na];
        rc = orc_cache_truncate(c, lc + na + 1);

        if (stage_log) {
            stage_log[2 * st.n_stages] = k;
            stage_log[2 * st.n_stages + 1] = na;
        }
        if (gamma_log)
            gamma_log[st.n_stages] = gamma;
        st.n_stages++;
        st.n_drafted += k;
        st.n_accepted += na;
        gamma = adapt_threshold(ad, k, na, &as, gamma);
    }
    st.n_emitted = emitted;
    if (stats)
        *stats = st;
    orc_cache_destroy(c);
    free(draft);
    free(rows);
    free(y);
    free(ymargin);
    return rc;
}

int orc_generate_sd(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new, const uint8_t *skip,
                    int32_t k_max, float gamma, int32_t *out, double *margin, orc_sd_stats *stats,
                    int32_t *stage_log, float *draft_pmax)
{
    return generate_sd(m, prompt, t, max_new, skip, k_max, gamma, NULL, out, margin, stats, stage_log, draft_pmax,
                       NULL);
}

int orc_generate_sd_adaptive(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                             const uint8_t *skip, int32_t k_max, const orc_adaptive *ad, int32_t *out,
                             double *margin, orc_sd_stats *stats, int32_t *stage_log, float *draft_pmax,
                             float *gamma_log)
{
    if (!ad || ad->gamma0 != ad->gamma0 || ad->alpha != ad->alpha || ad->epsilon != ad->epsilon ||
        ad->beta1 != ad->beta1 || ad->beta2 != ad->beta2)
        return -1;
    return generate_sd(m, prompt, t, max_new, skip, k_max, 0.0f, ad, out, margin, stats, stage_log, draft_pmax,
                       gamma_log);
}

/* ------------------------------------------------------------------------ */
/* Sampling variant (appendix: self-speculative decoding with random
 * sampling and the adaptive draft exit). */

/* Philox4x64-10, from its definition (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC'11): ten rounds of
 * (x0, x1, x2, x3) -> (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1,
 * lo(M0 x0)), with the key advanced by the Weyl constants between rounds. */
void orc_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
    const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        const unsigned __int128 p0 = (unsigned __int128)M0 * x0;
        const unsigned __int128 p1 = (unsigned __int128)M1 * x2;
        const uint64_t y0 = (uint64_t)(p1 >> 64) ^ x1 ^ k0;
        const uint64_t y1 = (uint64_t)p1;
        const uint64_t y2 = (uint64_t)(p0 >> 64) ^ x3 ^ k1;
        const uint64_t y3 = (uint64_t)p0;
        x0 = y0;
        x1 = y1;
        x2 = y2;
        x3 = y3;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

double orc_uniform(uint64_t seed, int64_t index, int32_t purpose, int64_t stage)
{
    const uint64_t ctr[4] = {(uint64_t)index, (uint64_t)(uint32_t)purpose, (uint64_t)stage, 0};
    const uint64_t key[2] = {seed, 0};
    uint64_t o[4];
    orc_philox4x64(ctr, key, o);
    return (double)(o[0] >> 40) * 0x1p-24;
}

typedef struct {
    int32_t id;
    double w;
} wtok;

static int wtok_order(const void *a, const void *b)
{
    const wtok *x = (const wtok *)a, *y = (const wtok *)b;
    if (x->w != y->w)
        return x->w > y->w ? -1 : 1;
    return (x->id > y->id) - (x->id < y->id);
}

int32_t orc_warp(const double *logits, int32_t V, double temperature, double top_p, double *pi, double *cut_margin)
{
    if (!logits || !pi || V < 1 || !(temperature > 0.0) || !(top_p > 0.0))
        return -1;
    double mx = -INFINITY;
    for (int32_t v = 0; v < V; ++v)
        if ((double)(float)logits[v] > mx)
            mx = (double)(float)logits[v];
    /* unnormalised weights exp((l - max) / T); the top token has weight 1 */
    double z = 0.0;
    for (int32_t v = 0; v < V; ++v) {
        pi[v] = exp(((double)(float)logits[v] - mx) / temperature);
        z += pi[v];
    }
    int32_t kept = V;
    double cm = INFINITY;
    if (top_p < 1.0) {
        wtok *ord = (wtok *)malloc(sizeof(wtok) * (size_t)V);
        if (!ord)
            return -3;
        for (int32_t v = 0; v < V; ++v) {
            ord[v].id = v;
            ord[v].w = pi[v];
        }
        qsort(ord, (size_t)V, sizeof(wtok), wtok_order);
        /* the nucleus: the shortest prefix of that order whose mass reaches top_p */
        const double target = top_p * z;
        double s = 0.0;
        kept = 0;
        while (kept < V) {
            const double before = s;
            s += ord[kept].w;
            ++kept;
            if (s >= target) {
                cm = fmin(target - before, s - target) / z;
                break;
            }
        }
        for (int32_t i = kept; i < V; ++i)
            pi[ord[i].id] = 0.0;
        free(ord);
    }
    double zs = 0.0;
    for (int32_t v = 0; v < V; ++v)
        zs += pi[v];
    for (int32_t v = 0; v < V; ++v)
        pi[v] /= zs;
    if (cut_margin)
        *cut_margin = cm;
    return kept;
}

/* Inverse-CDF draw in id order: the smallest x with u * W < w_0 + .. + w_x
 * (W the total weight); margin: the distance of u * W from the ends of x's
 * interval, relative to W. */
static int32_t draw(const double *w, int32_t V, double u, double *margin)
{
    double tot = 0.0;
    for (int32_t v = 0; v < V; ++v)
        tot += w[v];
    const double target = u * tot;
    double c = 0.0;
    int32_t last = 0;
    for (int32_t v = 0; v < V; ++v) {
        if (!(w[v] > 0.0))
            continue;
        const double before = c;
        c += w[v];
        last = v;
        if (target < c) {
            *margin = fmin(target - before, c - target) / tot;
            return v;
        }
    }
    *margin = 0.0; /* u * W reached the rounded total: the last token with weight */
    return last;
}

static int check_sampling(const orc_sampling *sp)
{
    return (sp && sp->temperature > 0.0 && sp->top_p > 0.0 && sp->top_p <= 1.0 && isfinite(sp->temperature)) ? 0
                                                                                                               : -1;
}

int orc_generate_ar_sample(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                           const orc_sampling *sp, int32_t *out, double *margin)
{
    if (!m || max_new < 0 || (max_new > 0 && !out) || check_prompt(m, prompt, t) || check_sampling(sp))
        return -1;
    const int32_t V = m->c.vocab;
    orc_cache *c = orc_cache_create(m, t + max_new + 1);
    double *lg = (double *)malloc(sizeof(double) * (size_t)V);
    double *pi = (double *)malloc(sizeof(double) * (size_t)V);
    if (!c || !lg || !pi) {
        orc_cache_destroy(c);
        free(lg);
        free(pi);
        return -3;
    }
    int rc = prefill(m, c, prompt, t);
    int32_t last = prompt[t - 1];
    /* token i ~ the warped full-model distribution given everything before it */
    for (int32_t i = 0; rc == 0 && i < max_new; ++i) {
        rc = orc_forward(m, c, &last, 1, NULL, lg, NULL, NULL, NULL);
        if (rc)
            break;
        double cm, dm;
        orc_warp(lg, V, sp->temperature, sp->top_p, pi, &cm);
        out[i] = draw(pi, V, orc_uniform(sp->seed, i, ORC_U_FINAL, i), &dm);
        if (margin)
            margin[i] = fmin(cm, dm);
        last = out[i];
    }
    orc_cache_destroy(c);
    free(lg);
    free(pi);
    return rc;
}

int orc_generate_sd_sample(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new,
                           const uint8_t *skip, int32_t k_max, float gamma, const orc_adaptive *ad,
                           const orc_sampling *sp, int32_t *out, double *margin, orc_sd_stats *stats,
                           int32_t *stage_log, float *draft_qmax, float *gamma_log)
{
    if (!m || max_new < 0 || (max_new > 0 && !out) || k_max < 0 || gamma != gamma || check_prompt(m, prompt, t) ||
        check_sampling(sp))
        return -1;
    if (ad && (ad->gamma0 != ad->gamma0 || ad->alpha != ad->alpha || ad->epsilon != ad->epsilon ||
               ad->beta1 != ad->beta1 || ad->beta2 != ad->beta2))
        return -1;
    if (skip)
        for (int i = 0; i < 2 * m->c.n_layers; ++i)
            if (skip[i] > 1)
                return -1;
    const int32_t V = m->c.vocab;
    const size_t K1 = (size_t)k_max + 1;
    adapt_state as = {0.0, ad ? ad->gamma0 : (double)gamma, 0};
    if (ad)
        gamma = (float)as.gamma_d;
    orc_sd_stats st;
    memset(&st, 0, sizeof st);
    st.min_gamma_gap = INFINITY;
    st.min_draft_margin = INFINITY;
    orc_cache *c = orc_cache_create(m, t + max_new + k_max + 1);
    int32_t *draft = (int32_t *)malloc(sizeof(int32_t) * K1);
    int32_t *rows = (int32_t *)malloc(sizeof(int32_t) * K1);
    double *dmarg = (double *)malloc(sizeof(double) * K1);      /* draw margin of each draft */
    double *qcut = (double *)malloc(sizeof(double) * K1);       /* top-p cut margins, draft rows */
    double *pcut = (double *)malloc(sizeof(double) * K1);       /* and verification rows */
    double *q = (double *)malloc(sizeof(double) * K1 * (size_t)V);  /* warped draft distributions */
    double *p = (double *)malloc(sizeof(double) * K1 * (size_t)V);  /* warped full-model distributions */
    double *lg = (double *)malloc(sizeof(double) * K1 * (size_t)V);
    if (!c || !draft || !rows || !dmarg || !qcut || !pcut || !q || !p || !lg) {
        orc_cache_destroy(c);
        free(draft);
        free(rows);
        free(dmarg);
        free(qcut);
        free(pcut);
        free(q);
        free(p);
        free(lg);
        return -3;
    }
    int rc = prefill(m, c, prompt, t);
    int32_t last = prompt[t - 1];
    int32_t emitted = 0;

    while (rc == 0 && emitted < max_new) {
        const int64_t stage = st.n_stages;
        const int32_t lc = c->len;
        const int32_t kcap = stage_budget(k_max, max_new, emitted);

        /* Drafting: each draft is drawn from the warped draft distribution;
         * the stage stops after a draft whose warped maximum is below gamma
         * (that draft is still verified). */
        int32_t k = 0;
        for (int32_t j = 0; j < kcap; ++j) {
            int32_t in = j > 0 ? draft[j - 1] : last;
            rc = orc_forward(m, c, &in, 1, skip, lg, NULL, NULL, NULL);
            if (rc)
                break;
            double *qj = q + (size_t)j * V;
            orc_warp(lg, V, sp->temperature, sp->top_p, qj, &qcut[j]);
            double qmax = 0.0;
            for (int32_t v = 0; v < V; ++v)
                if (qj[v] > qmax)
                    qmax = qj[v];
            draft[j] = draw(qj, V, orc_uniform(sp->seed, emitted + j, ORC_U_DRAFT, stage), &dmarg[j]);
            const float qf = (float)qmax;
            if (draft_qmax)
                draft_qmax[st.n_draft_steps] = qf;
            st.n_draft_steps++;
            const double gap = fabs((double)qf - (double)gamma);
            if (gap < st.min_gamma_gap)
                st.min_gamma_gap = gap;
            k = j + 1;
            if (qf < gamma)
                break;
        }
        if (rc)
            break;

        /* Verification: one full-model forward over [last, d_1 .. d_k]. */
        rc = orc_cache_truncate(c, lc);
        if (rc)
            break;
        rows[0] = last;
        for (int32_t j = 0; j < k; ++j)
            rows[j + 1] = draft[j];
        rc = orc_forward(m, c, rows, k + 1, NULL, lg, NULL, NULL, NULL);
        if (rc)
            break;
        for (int32_t i = 0; i <= k; ++i)
            orc_warp(lg + (size_t)i * V, V, sp->temperature, sp->top_p, p + (size_t)i * V, &pcut[i]);

        /* Draft i is accepted when r < min(1, p_i(d) / q_i(d)); the first
         * rejection ends the stage. */
        int32_t na = 0;
        double reject_margin = INFINITY;
        for (; na < k; ++na) {
            const int32_t d = draft[na];
            const double r = orc_uniform(sp->seed, emitted + na, ORC_U_ACCEPT, stage);
            const double ratio = p[(size_t)na * V + d] / q[(size_t)na * V + d];
            const double lim = ratio < 1.0 ? ratio : 1.0;
            const double am = fabs(r - lim);
            if (!(r < lim)) {
                reject_margin = am;
                break;
            }
            const double mg = fmin(fmin(dmarg[na], am), fmin(qcut[na], pcut[na]));
            if (margin)
                margin[emitted + na] = mg;
            out[emitted + na] = d;
        }
        /* The token after the accepted drafts: at a rejection, a draw from
         * max(0, p - q) normalised (from p if that is empty); after a fully
         * accepted stage, a draw from p. */
        const double uf = orc_uniform(sp->seed, emitted + na, ORC_U_FINAL, stage);
        double fm, mg;
        int32_t y;
        const double *pn = p + (size_t)na * V;
        if (na < k) {
            const double *qn = q + (size_t)na * V;
            double *res = lg; /* logits no longer needed */
            double tot = 0.0;
            for (int32_t v = 0; v < V; ++v) {
                res[v] = pn[v] > qn[v] ? pn[v] - qn[v] : 0.0;
                tot += res[v];
            }
            y = tot > 0.0 ? draw(res, V, uf, &fm) : draw(pn, V, uf, &fm);
            mg = fmin(fmin(fm, reject_margin), fmin(qcut[na], pcut[na]));
        } else {
            y = draw(pn, V, uf, &fm);
            mg = fmin(fm, pcut[na]);
        }
        if (margin)
            margin[emitted + na] = mg;
        out[emitted + na] = y;
        emitted += na + 1;
        last = y;
        rc = orc_cache_truncate(c, lc + 1 + na);

        if (stage_log) {
            stage_log[2 * st.n_stages] = k;
            stage_log[2 * st.n_stages + 1] = na;
        }
        if (gamma_log)
            gamma_log[st.n_stages] = gamma;
        st.n_stages++;
        st.n_drafted += k;
        st.n_accepted += na;
        gamma = adapt_threshold(ad, k, na, &as, gamma); /* the same rule as the greedy form */
    }
    st.n_emitted = emitted;
    if (stats)
        *stats = st;
    orc_cache_destroy(c);
    free(draft);
    free(rows);
    free(dmarg);
    free(qcut);
    free(pcut);
    free(q);
    free(p);
    free(lg);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* FP8 draft weights.  The adaptation appendix (Quantization subsection and
 * table) runs self-speculative decoding on LLM.int8() FP8/FP4 weights to cut
 * memory.  Here only a copy of the draft's weights is quantized, to stream
 * half the bytes per draft step; the verification keeps the stored bf16
 * weights, so the emitted tokens are still exactly those of greedy decoding
 * of the original model, and only the drafts (hence the stage trace) follow
 * the quantized copy.
 *
 * Format: OCP FP8 E4M3 (1 sign bit, 4 exponent bits with bias 7, 3 mantissa
 * bits; exponent field 0 subnormal; S.1111.111 NaN; largest value 448), one
 * power-of-two scale 2^e per output row: e is the smallest integer with
 * max_k |W[n][k]| * 2^-e <= 448, so scaling is exact and the stored byte is
 * the nearest E4M3 value (ties to even) of W[n][k] * 2^-e. */

double orc_fp8_value(uint8_t b)
{
    const int sgn = b >> 7, f = (b >> 3) & 15, mt = b & 7;
    if (f == 15 && mt == 7)
        return NAN;
    const double v = f == 0 ? ldexp((double)mt, -9) : ldexp(1.0 + (double)mt / 8.0, f - 7);
    return sgn ? -v : v;
}

/* The byte of the nearest E4M3 value (ties to even) of v, |v| <= 448. */
static uint8_t fp8_encode(double v)
{
    const uint8_t sgn = signbit(v) ? 0x80 : 0;
    const double a = fabs(v);
    if (a == 0.0)
        return sgn;
    int e;
    (void)frexp(a, &e); /* a = f 2^e, 0.5 <= f < 1: floor(log2 a) = e - 1 */
    const int quantum = e - 1 < -6 ? -9 : e - 1 - 3;
    const double r = ldexp(rint(ldexp(a, -quantum)), quantum); /* rint: to nearest, ties to even */
    if (r == 0.0)
        return sgn;
    (void)frexp(r, &e);
    const int ex = e - 1;
    if (ex < -6)
        return sgn | (uint8_t)ldexp(r, 9);
    return sgn | (uint8_t)((ex + 7) << 3) | (uint8_t)(ldexp(r, -ex) * 8.0 - 8.0);
}

/* The smallest e with amax * 2^-e <= 448 = 0.875 * 2^9; 0 for amax = 0. */
static int32_t fp8_row_exponent(double amax)
{
    if (amax == 0.0)
        return 0;
    int e;
    const double f = frexp(amax, &e);
    return e - 9 + (f > 0.875 ? 1 : 0);
}

int orc_quantize_fp8_rows(const uint16_t *w, int64_t n_rows, int64_t n_cols, uint8_t *q, int32_t *e)
{
    if (!w || !q || !e || n_rows < 0 || n_cols < 1)
        return -1;
    for (int64_t n = 0; n < n_rows; ++n) {
        double amax = 0.0;
        for (int64_t k = 0; k < n_cols; ++k) {
            const double a = fabs(bf16_to_double(w[n * n_cols + k]));
            if (a > amax)
                amax = a;
        }
        e[n] = fp8_row_exponent(amax);
        for (int64_t k = 0; k < n_cols; ++k)
            q[n * n_cols + k] = fp8_encode(ldexp(bf16_to_double(w[n * n_cols + k]), -e[n]));
    }
    return 0;
}

static void free_draft_fp8(orc_model *m)
{
    for (int k = 0; k < FP8_KINDS; ++k) {
        for (int l = 0; m->fp8_q[k] && l < m->c.n_layers; ++l) {
            free(m->fp8_q[k][l]);
            free(m->fp8_e[k][l]);
        }
        free(m->fp8_q[k]);
        free(m->fp8_e[k]);
        m->fp8_q[k] = NULL;
        m->fp8_e[k] = NULL;
    }
}

int orc_set_draft_fp8(orc_model *m, const uint8_t *skip)
{
    if (!m || m->c.wdtype != 1)
        return -1;
    free_draft_fp8(m);
    if (!skip)
        return 0;
    const int L = m->c.n_layers, d = m->c.d_model, hd = m->c.n_heads * m->c.head_dim, F = m->c.ffn_dim;
    const int64_t nqkv = (int64_t)(m->c.n_heads + 2 * m->c.n_kv_heads) * m->c.head_dim;
    for (int i = 0; i < 2 * L; ++i)
        if (skip[i] > 1)
            return -1;
    for (int k = 0; k < FP8_KINDS; ++k) {
        m->fp8_q[k] = (uint8_t **)calloc((size_t)L, sizeof(uint8_t *));
        m->fp8_e[k] = (int32_t **)calloc((size_t)L, sizeof(int32_t *));
        if (!m->fp8_q[k] || !m->fp8_e[k]) {
            free_draft_fp8(m);
            return -3;
        }
    }
    for (int l = 0; l < L; ++l) {
        const void *w[FP8_KINDS] = {m->w_qkv[l], m->w_o[l], m->w_gate_up[l], m->w_down[l]};
        const int64_t rows[FP8_KINDS] = {nqkv, d, 2 * (int64_t)F, d};
        const int64_t cols[FP8_KINDS] = {d, hd, d, F};
        for (int k = 0; k < FP8_KINDS; ++k) {
            const int run = k < FP8_GATE_UP ? !skip[2 * l] : !skip[2 * l + 1];
            if (!run)
                continue;
            m->fp8_q[k][l] = (uint8_t *)malloc((size_t)(rows[k] * cols[k]));
            m->fp8_e[k][l] = (int32_t *)malloc(sizeof(int32_t) * (size_t)rows[k]);
            if (!m->fp8_q[k][l] || !m->fp8_e[k][l]) {
                free_draft_fp8(m);
                return -3;
            }
            orc_quantize_fp8_rows((const uint16_t *)w[k], rows[k], cols[k], m->fp8_q[k][l], m->fp8_e[k][l]);
        }
    }
    return 0;
}
