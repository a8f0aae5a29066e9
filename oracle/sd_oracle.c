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

struct orc_model {
    orc_config c;
    const void *tok_emb, *final_norm, *lm_head;
    const void **attn_norm, **w_qkv, **w_o, **mlp_norm, **w_gate_up, **w_down;
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

void orc_destroy(orc_model *m)
{
    if (!m)
        return;
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
            linear(m, m->w_qkv[l], nqkv, d, u, n, qkv);
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
            linear(m, m->w_o[l], d, (int64_t)H * dh, o, n, t);
            for (int64_t i = 0; i < (int64_t)n * d; ++i)
                h[i] += t[i];
        }
        if (!(skip && skip[2 * l + 1])) {
            for (int r = 0; r < n; ++r)
                rmsnorm(m, m->mlp_norm[l], h + (int64_t)r * d, u + (int64_t)r * d);
            linear(m, m->w_gate_up[l], 2 * (int64_t)F, d, u, n, gu);
            for (int r = 0; r < n; ++r)
                for (int f = 0; f < F; ++f) {
                    const double *gr = gu + (int64_t)r * 2 * F;
                    mm[(int64_t)r * F + f] = silu(gr[f]) * gr[F + f];
                }
            linear(m, m->w_down[l], d, F, mm, n, t);
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

/* Self-speculative decoding; ad == NULL keeps the threshold fixed at gamma,
 * otherwise it starts at ad->gamma0 and follows Eqs. 2-4. */
static int generate_sd(orc_model *m, const int32_t *prompt, int32_t t, int32_t max_new, const uint8_t *skip,
                       int32_t k_max, float gamma, const orc_adaptive *ad, int32_t *out, double *margin,
                       orc_sd_stats *stats, int32_t *stage_log, float *draft_pmax, float *gamma_log)
{
    if (!m || max_new < 0 || (max_new > 0 && !out) || k_max < 0 || gamma != gamma || check_prompt(m, prompt, t))
        return -1;
    /* threshold state of the adaptive rule: gamma_d is the threshold in
     * float64, the exit test uses it rounded to float32 */
    double gamma_d = ad ? ad->gamma0 : (double)gamma;
    double ar = 0.0;
    int64_t n_updates = 0;
    if (ad)
        gamma = (float)gamma_d;
    if (skip)
        for (int i = 0; i < 2 * m->c.n_layers; ++i)
            if (skip[i] > 1)
                return -1;
    orc_sd_stats st;
    memset(&st, 0, sizeof st);
    st.min_gamma_gap = INFINITY;
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
        /* Reading: at most K drafts per stage, and never more than the
         * tokens still to emit minus the one the verification adds. */
        int32_t kcap = k_max;
        if (kcap > max_new - emitted - 1)
            kcap = max_new - emitted - 1;

        /* Drafting stage: greedy tokens of the model with the skip set
         * bypassed; exit right after a token whose top-1 probability is
         * below gamma (that token is still verified). */
        int32_t k = 0;
        for (int32_t j = 0; j < kcap; ++j) {
            int32_t in = j == 0 ? last : draft[j - 1];
            float p;
            rc = orc_forward(m, c, &in, 1, skip, NULL, &draft[j], &p, NULL);
            if (rc)
                break;
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

        /* Adaptive threshold, after the verification stage (Eqs. 2-4): the
         * stage's acceptance rate AR_e = n_e / k_e is smoothed into AR
         * (AR = AR_e at the first stage), the threshold moves by epsilon up
         * when AR is at most the target alpha and down otherwise, and the
         * move is smoothed by beta2.  Reading: a stage without drafts
         * (k_e = 0, only at the end of generation or with K = 0) says
         * nothing about acceptance and leaves AR and gamma as they are. */
        if (ad && k > 0) {
            const double ar_e = (double)na / (double)k;
            ar = n_updates == 0 ? ar_e : ad->beta1 * ar + (1.0 - ad->beta1) * ar_e;
            n_updates++;
            const double gamma_t = ar <= ad->alpha ? gamma_d + ad->epsilon : gamma_d - ad->epsilon;
            gamma_d = ad->beta2 * gamma_d + (1.0 - ad->beta2) * gamma_t;
            gamma = (float)gamma_d;
        }
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
