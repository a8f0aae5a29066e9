// Host orchestration behind the C ABI of include/sd.h: model and cache
// objects, the decoder forward as a sequence of kernel launches, and the
// two decoding loops (greedy autoregressive, Algorithm 1; greedy
// self-speculative, Algorithm 2 with the static draft exit of Sec. 3.4).
#include "sd.h"
#include "sd_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "host_api.h"

#if defined(__x86_64__)
#include <immintrin.h>
#endif

using namespace sdk;

namespace {

thread_local std::string g_err;

sd_status fail(sd_status st, const std::string &msg) {
    g_err = msg;
    return st;
}

#define SD_HIP(expr)                                                                                   \
    do {                                                                                               \
        hipError_t e_ = (expr);                                                                        \
        if (e_ != hipSuccess)                                                                          \
            return fail(SD_ERR_DEVICE, std::string(#expr) + " failed: " + hipGetErrorString(e_));     \
    } while (0)

#define SD_TRY(expr)                                                                                   \
    do {                                                                                               \
        sd_status s_ = (expr);                                                                         \
        if (s_ != SD_OK)                                                                               \
            return s_;                                                                                 \
    } while (0)

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

enum LinearKind { LK_QKV = 0, LK_O = 1, LK_GATE_UP = 2, LK_DOWN = 3, LK_HEAD = 4, LK_COUNT = 5 };

// Event pairs timing the steps of a self-speculative decode (a ring; at
// most four steps are unread at a time).
constexpr int STEP_EVENT_PAIRS = 8;

// Forwards of the timed regime per forward whose launches the measurement
// hook brackets with events.
constexpr int64_t TIMED_SAMPLE = 16;

// How one linear layer is launched for one row regime.
struct Plan {
    int kind;     // LinearKind
    int regime;   // 1, 2 or 16: the row counts the plan serves
    int path;     // LinearPath
    int rows;     // weight rows per work-group
    int n_tiles;  // GEMV/VALU: work-groups; MFMA: 16-row tiles
    int waves;    // MFMA: waves per work-group splitting the reduction
    int splits;   // MFMA output projections: split-K partials folded by the next norm
    int chunks;   // PATH_WAVE2: loads in flight per wave (0: the path's default)
    int N, K, epi;
};

// Scratch of one decode-path forward (up to MAX_ROWS rows): the residual
// stream, the attention and MLP activations, split-K and attention
// partials, the lm-head partials and the control block.  A model owns one
// (allocated at creation); the allocation-free forward carves another out
// of a static device array.
struct Workspace {
    float *h = nullptr, *q = nullptr, *o = nullptr, *mbuf = nullptr;
    float *part = nullptr;  // split-K partials of the MFMA output projections
    float *ssq = nullptr;   // sums of h^2 per row and slice for the next normed MFMA layer
    // MFMA-path activations split into X_TERMS bf16 terms in fragment layout
    // (48 xld elements each): xa holds normalised inputs and the attention
    // output, xb the SwiGLU output.
    uint16_t *xa = nullptr, *xb = nullptr;
    int64_t xld = 0;
    float4 *head_part = nullptr;
    float *attn_o = nullptr;    // [splits][n_heads][MAX_ROWS][head_dim]
    float2 *attn_ml = nullptr;  // [splits][n_heads][MAX_ROWS]
    DevCtl *ctl = nullptr;
};

}  // namespace

struct sd_kv_cache {
    sd_model *model;
    void *buf;
    bool owns;
    int32_t cap;
    int32_t len;
};

struct sd_model {
    sd_config cfg{};
    bool bf16 = false;
    size_t wsize = 4;
    const void *tok_emb = nullptr, *final_norm = nullptr, *lm_head = nullptr;
    std::vector<const void *> attn_norm, w_qkv, w_o, mlp_norm, w_gate_up, w_down;
    hipStream_t stream = nullptr;

    Plan plan1[LK_COUNT];  // one row (draft / autoregressive step)
    Plan plan2[LK_COUNT];  // up to 2 rows (verification of one draft)
    Plan planm[LK_COUNT];  // up to 16 rows (longer verification, prefill)
    Workspace ws;           // scratch of the decode-path forwards
    int max_head_tiles = 1; // lm-head tiles of the widest plan
    // FP8 copies of the draft's weights (sd_model_quantize_draft), per layer
    // and kind (QKV, O, gate/up, down): E4M3 bytes and row exponents, or null
    std::vector<std::array<uint8_t *, 4>> fp8_q;
    std::vector<std::array<int32_t *, 4>> fp8_e;
    bool has_fp8 = false;
    // sampling variant: logits of the verification / autoregressive rows and
    // of the stage's drafts, the rows' nucleus statistics, the parameters
    float *slog_v = nullptr, *slog_d = nullptr;
    RowStat *svstat = nullptr, *sdstat = nullptr;
    SampleParams sp_cur{};
    int attn_splits_cap = 0;  // key chunks ws.attn_o / ws.attn_ml hold
    float2 *rope = nullptr;
    int rope_cap = 0;
    // large-M forward (bfloat16 models): residual stream, GEMM output,
    // rotated queries, and the GEMM inputs as X_TERMS terms, PF_ROWS rows each
    bool pf_ok = false;
    float *pf_h = nullptr, *pf_c = nullptr, *pf_q = nullptr, *pf_part = nullptr;
    uint16_t *pf_x = nullptr;  // terms of the GEMM inputs: normed rows, attention output
    int64_t pf_term = 0;
    uint16_t *pf_y = nullptr;  // terms of the MLP activation: the gate/up GEMM's output, the down GEMM's input
    int64_t pf_y_term = 0;
    DevState *st = nullptr;
    Mailbox *mb_host = nullptr;
    Mailbox *mb_dev = nullptr;
    int32_t *d_tokens = nullptr;
    int d_tokens_cap = 0;
    int32_t *d_out = nullptr;
    int d_out_cap = 0;
    int32_t *d_log = nullptr;  // (k_e, n_e) pairs
    int d_log_cap = 0;         // int32 elements
    float *d_glog = nullptr;   // threshold of each stage
    int d_glog_cap = 0;
    sd_kv_cache *gen_cache = nullptr;
    std::vector<sd_kv_cache *> caches;  // caller-created caches, detached on destroy
    // ev[0], ev[1]: prefill; then STEP_EVENT_PAIRS pairs for the decode steps
    hipEvent_t ev[2 + 2 * STEP_EVENT_PAIRS] = {};
    // measurement hook (sd_model_time_kernel)
    int timed_kind = -1, timed_regime = 0;
    int64_t timed_forwards = 0;  // forwards of the timed regime since the hook was set
    bool timed_now = false;      // this forward's launches of the timed class are bracketed
    int timed_rows_lo = 0, timed_rows_hi = 0;  // row bounds seen by the timed launches
    std::vector<hipEvent_t> tev;  // pairs
    size_t tev_used = 0;
    int64_t timed_launches = 0;
    double timed_ms = 0.0;
};

namespace {

int cdiv(int a, int b) { return (a + b - 1) / b; }

// Elements per term of the MFMA-path activation buffers (xa, xb).
int64_t xld_of(const sd_config &c) {
    return std::max<int64_t>({c.d_model, (int64_t)c.n_heads * c.head_dim, c.ffn_dim});
}

// Tile rows for the QKV layer must hold whole rotary pairs of one head.
int qkv_gemv_rows(int head_dim, int want) {
    const int half = head_dim / 2;
    for (int r = want; r >= 4; r /= 2)
        if (half % (r / 2) == 0)
            return r;
    return 4;
}

bool mfma_ok(const sd_model *m, LinearKind kind) {
    const sd_config &c = m->cfg;
    const int K = kind == LK_O ? c.n_heads * c.head_dim : (kind == LK_DOWN ? c.ffn_dim : c.d_model);
    return m->bf16 && K % 128 == 0 && (kind != LK_QKV || (c.head_dim / 2) % 8 == 0);
}

// rows: the largest row count the plan serves (1, 2 or 16).  Tile sizes
// follow measurements at the 13B shape.
Plan make_plan(const sd_model *m, LinearKind kind, int rows) {
    const sd_config &c = m->cfg;
    Plan p{};
    p.kind = kind;
    p.regime = rows;
    p.waves = 4;
    p.splits = 1;
    switch (kind) {
    case LK_QKV:
        p.N = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
        p.K = c.d_model;
        p.epi = EPI_QKV;
        break;
    case LK_O:
        p.N = c.d_model;
        p.K = c.n_heads * c.head_dim;
        p.epi = EPI_RESID;
        break;
    case LK_GATE_UP:
        p.N = 2 * c.ffn_dim;
        p.K = c.d_model;
        p.epi = EPI_SWIGLU;
        break;
    case LK_DOWN:
        p.N = c.d_model;
        p.K = c.ffn_dim;
        p.epi = EPI_RESID;
        break;
    default:
        p.N = c.vocab;
        p.K = c.d_model;
        p.epi = EPI_HEAD;
        break;
    }
    // Two rows (one-draft verification) of a bf16 model: every layer on
    // one-wave VALU tiles, 8 weight rows for the wide layers and 4 for the
    // output projections.  Measured at the 13B shape against the earlier
    // plan (MFMA for QKV and the lm-head, four-wave tiles otherwise): QKV
    // 30.2 against 31.6 us, gate/up 49.0 against 50.0, O 11.8 against 13.0,
    // down 25.6 against 27.8, lm-head 54.6 against 58.6.
    if (rows == 2 && m->bf16) {
        p.path = PATH_WAVE2;
        p.rows = kind == LK_QKV ? qkv_gemv_rows(c.head_dim, 8) : ((kind == LK_O || kind == LK_DOWN) ? 4 : 8);
        // Shapes where another tile measured faster: the 70B output and down
        // projections with one chunk's loads in flight (standalone 24.5
        // against 25.8 us and 76.9 against 81.9; the 70B two-row
        // verification 24.37 -> 22.66 ms).  At 7B neither 4-row QKV and
        // gate/up tiles (standalone 21.5 against 23.9 us, 35.1 against 36.2)
        // nor one chunk in flight for O and down made the verification
        // faster (2.98 -> 3.03 and 3.10 ms), so it keeps these defaults.
        struct Tuned {
            int kind, N, K, rows, chunks;
        };
        static const Tuned tuned[] = {{LK_O, 8192, 8192, 4, 1}, {LK_DOWN, 8192, 28672, 4, 1}};
        for (const Tuned &t : tuned) {
            const bool fits = kind != LK_QKV || qkv_gemv_rows(c.head_dim, t.rows) == t.rows;
            if (t.kind == kind && t.N == p.N && t.K == p.K && fits) {
                p.rows = t.rows;
                p.chunks = t.chunks;
            }
        }
        if (kind == LK_QKV)
            p.n_tiles = (c.n_heads + 2 * c.n_kv_heads) * ((c.head_dim / 2) / (p.rows / 2));
        else if (kind == LK_GATE_UP)
            p.n_tiles = cdiv(c.ffn_dim, p.rows / 2);
        else
            p.n_tiles = cdiv(p.N, p.rows);
        return p;
    }
    if (rows > 2 && mfma_ok(m, kind)) {
        p.path = PATH_MFMA;
        if (kind == LK_QKV)
            p.n_tiles = (c.n_heads + 2 * c.n_kv_heads) * ((c.head_dim / 2) / 8);
        else if (kind == LK_GATE_UP)
            p.n_tiles = cdiv(c.ffn_dim, 8);
        else
            p.n_tiles = cdiv(p.N, 16);
        // 16-row tiles; the work-group shape is picked per launch from the
        // packing count (mfma_shape_tn / mfma_shape_nw)
        p.rows = 16;
        if (kind == LK_O || kind == LK_DOWN) {
            // Narrow outputs: the reduction is split over work-groups and the
            // partial sums are folded into the residual stream by the norm
            // that reads it next (all readers of the residual stream must
            // then be MFMA layers).
            const bool fold = mfma_ok(m, LK_QKV) && mfma_ok(m, LK_GATE_UP) && mfma_ok(m, LK_HEAD);
            if (fold) {
                p.epi = EPI_PARTIAL;
                p.splits = p.K >= 8192 ? 8 : 4;
            }
        }
        return p;
    }
    p.path = rows == 1 ? PATH_GEMV : (rows <= 2 ? PATH_VALU2 : PATH_VALU16);
    // weight rows per work-group: 8 for the wide layers of the one-row GEMV,
    // 4 otherwise (the QKV tile also holds whole rotary pairs)
    const int wide = (rows == 1 || (rows == 2 && kind == LK_GATE_UP)) ? 8 : 4;
    if (kind == LK_QKV) {
        p.rows = qkv_gemv_rows(c.head_dim, rows <= 2 ? 8 : 4);
        p.n_tiles = (c.n_heads + 2 * c.n_kv_heads) * ((c.head_dim / 2) / (p.rows / 2));
    } else if (kind == LK_GATE_UP) {
        p.rows = wide;
        p.n_tiles = cdiv(c.ffn_dim, wide / 2);
    } else if (kind == LK_HEAD) {
        p.rows = wide;
        p.n_tiles = cdiv(p.N, wide);
    } else {
        p.rows = 4;
        p.n_tiles = cdiv(p.N, p.rows);
    }
    return p;
}

int head_tiles(const Plan &p) { return p.n_tiles; }

template <typename T>
sd_status dev_alloc(T **p, size_t count) {
    *p = nullptr;
    if (count == 0)
        count = 1;
    if (hipMalloc(reinterpret_cast<void **>(p), count * sizeof(T)) != hipSuccess) {
        *p = nullptr;
        return fail(SD_ERR_OOM, "device allocation of " + std::to_string(count * sizeof(T)) + " bytes failed");
    }
    return SD_OK;
}

void dev_free(void *p) {
    if (p)
        (void)hipFree(p);
}

// Rotary table for positions [0, cap): (cos, sin) of pos * base^(-2i/dh),
// computed in double and rounded to float.
sd_status ensure_rope(sd_model *m, int cap) {
    if (cap <= m->rope_cap)
        return SD_OK;
    const int half = m->cfg.head_dim / 2;
    std::vector<float2> tab((size_t)cap * half);
    for (int p = 0; p < cap; ++p)
        for (int i = 0; i < half; ++i) {
            const double theta = std::pow((double)m->cfg.rope_base, -2.0 * (double)i / (double)m->cfg.head_dim);
            const double ang = (double)p * theta;
            tab[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
        }
    SD_HIP(hipStreamSynchronize(m->stream));
    float2 *nt = nullptr;
    SD_TRY(dev_alloc(&nt, tab.size()));
    if (hipMemcpy(nt, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess) {
        dev_free(nt);
        return fail(SD_ERR_DEVICE, "rotary table upload failed");
    }
    dev_free(m->rope);
    m->rope = nt;
    m->rope_cap = cap;
    return SD_OK;
}

int attn_chunk_min_of(const sd_model *m) {
    return attn_chunk_min(m->bf16, m->cfg.head_dim, m->cfg.n_heads, m->cfg.n_kv_heads);
}

sd_status ensure_attn(sd_model *m, int cap) {
    const int splits = attn_split_slots(cap, attn_chunk_min_of(m));
    if (splits <= m->attn_splits_cap)
        return SD_OK;
    SD_HIP(hipStreamSynchronize(m->stream));
    float *po = nullptr;
    float2 *pml = nullptr;
    const size_t slots = (size_t)splits * m->cfg.n_heads * MAX_ROWS;
    SD_TRY(dev_alloc(&po, slots * m->cfg.head_dim));
    if (dev_alloc(&pml, slots) != SD_OK) {
        dev_free(po);
        return SD_ERR_OOM;
    }
    dev_free(m->ws.attn_o);
    dev_free(m->ws.attn_ml);
    m->ws.attn_o = po;
    m->ws.attn_ml = pml;
    m->attn_splits_cap = splits;
    return SD_OK;
}

template <typename T>
sd_status ensure_buf(sd_model *m, T **buf, int *cap, int need) {
    if (need <= *cap)
        return SD_OK;
    SD_HIP(hipStreamSynchronize(m->stream));
    T *nb = nullptr;
    SD_TRY(dev_alloc(&nb, (size_t)need));
    dev_free(*buf);
    *buf = nb;
    *cap = need;
    return SD_OK;
}

sd_status launch(hipError_t e, const char *what) {
    if (e != hipSuccess)
        return fail(SD_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
    return SD_OK;
}

// One linear layer over up to max_rows rows.  X (float32, with the RMSNorm
// gain folded in by the VALU kernels) feeds the VALU paths; the MFMA path
// reads the bf16 term planes xs (g * h from k_prep_norm, the layer dividing
// by rms(h) itself, or split by the producer for the output projections).
sd_status run_linear(sd_model *m, const Workspace &w, const Plan &p, int max_rows, const void *W, const float *X,
                     int64_t ldx, const void *gain, const EpiArgs &epi, const uint16_t *xs, bool guarded = false,
                     const int32_t *wexp = nullptr) {
    LinearArgs a{};
    a.guarded = guarded ? 1 : 0;
    a.wexp = wexp;
    a.W = W;
    a.N = p.N;
    a.K = p.K;
    if (p.path == PATH_MFMA) {
        a.Xs = xs;
        a.max_rows = max_rows;
        if (gain) {  // the fragments hold g * h; 1/rms(h) from the slices' sums
            a.ssq = w.ssq;
            a.ssq_slices = prep_slices(p.K);
        }
    } else {
        a.X = X;
        a.ldx = ldx;
        a.gain = gain;
    }
    a.eps = m->cfg.rms_eps;
    a.ctl = w.ctl;
    a.epi = epi;
    a.waves = p.waves;
    a.splits = p.splits;
    a.part = w.part;
    a.n_tiles = p.n_tiles;
    const bool timed = m->timed_now && p.kind == m->timed_kind && p.regime == m->timed_regime &&
                       p.path != PATH_GEMV_FP8 && m->tev_used + 2 <= 2 * 65536;
    if (timed) {
        if (m->tev_used + 2 > m->tev.size()) {
            for (int i = 0; i < 256; ++i) {
                hipEvent_t e;
                SD_HIP(hipEventCreate(&e));
                m->tev.push_back(e);
            }
        }
        m->timed_rows_lo = m->timed_rows_lo ? std::min(m->timed_rows_lo, max_rows) : max_rows;
        m->timed_rows_hi = std::max(m->timed_rows_hi, max_rows);
    }
    LaunchTiming lt;
    if (timed) {
        lt.start = m->tev[m->tev_used];
        lt.stop = m->tev[m->tev_used + 1];
    }
    SD_TRY(launch(launch_linear(a, p.epi, m->bf16, p.path, p.rows, p.n_tiles, m->stream, lt, p.chunks),
                  "linear layer"));
    if (timed)
        m->tev_used += 2;
    if (p.epi == EPI_HEAD && epi.head.sampled) {
        SampleArgs sa{};
        sa.sp = m->sp_cur;
        sa.vocab = m->cfg.vocab;
        sa.ctl = w.ctl;
        sa.vlog = m->slog_v;
        sa.dlog = m->slog_d;
        sa.vstat = m->svstat;
        sa.dstat = m->sdstat;
        sa.head = epi.head;
        SD_TRY(launch(launch_sample_step(sa, max_rows, m->stream), "sampling step"));
    } else if (p.epi == EPI_HEAD) {
        SD_TRY(launch(launch_head_finalize(a, p.n_tiles, m->stream), "head finalize"));
    }
    return SD_OK;
}

// The MFMA operand of a normed layer into xa (MFMA path only), after folding
// the pending split-K partials of the last output projection: g * h, with
// the sums of h^2 per slice in ssq for the layer's 1/rms(h).
sd_status prep_norm(sd_model *m, const Workspace &w, const Plan &p, const void *gain, int &pending) {
    if (p.path != PATH_MFMA)
        return SD_OK;
    SD_TRY(launch(launch_prep_norm(w.h, m->cfg.d_model, gain, m->bf16, p.K, w.ctl, w.xa, w.part, pending, w.ssq,
                                   m->stream),
                  "norm"));
    pending = 0;
    return SD_OK;
}

struct HeadSpec {
    int mode = HEAD_NONE;
    float *logits = nullptr;
    bool run = false;
    bool sampled = false;  // sampling variant (parameters in sd_model::sp_cur)
};

// One decoder forward over the rows described by the device control block,
// enqueued in pieces: forward_begin (embedding), forward_layers (layers up
// to a bound; several calls continue one forward), forward_head.  max_rows
// (known to the host) bounds the row count and picks the kernels; skip is a
// host mask or null.
struct ForwardCursor {
    const Plan *P = nullptr;
    int max_rows = 0;
    int next_layer = 0;
    int pending = 0;       // split-K partials not yet folded into h
    bool guarded = false;  // launches may find the step cancelled (ctl->m = 0)
};

sd_status forward_begin(sd_model *m, const Workspace &w, int max_rows, ForwardCursor *cur) {
    const Plan *P = max_rows <= 1 ? m->plan1 : (max_rows <= 2 ? m->plan2 : m->planm);
    // The measurement hook times the class in one of every TIMED_SAMPLE
    // forwards of its regime, with events the runtime attaches to the
    // dispatch (the kernel's own start and end).
    m->timed_now = P[0].regime == m->timed_regime && m->timed_kind >= 0 &&
                   (m->timed_forwards++ % TIMED_SAMPLE) == 0;
    *cur = ForwardCursor{};
    cur->P = P;
    cur->max_rows = max_rows;
    return launch(launch_embed(m->tok_emb, m->bf16, m->cfg.d_model, w.ctl, w.h, m->cfg.d_model, m->stream),
                  "embedding");
}

sd_status forward_layers(sd_model *m, const Workspace &w, void *kv, int32_t cap, const uint8_t *skip,
                         ForwardCursor *cur, int layer_end) {
    const sd_config &c = m->cfg;
    const Plan *P = cur->P;
    const int max_rows = cur->max_rows;
    int &pending = cur->pending;
    const int64_t ldh = c.d_model, ldq = (int64_t)c.n_heads * c.head_dim;
    const size_t ksz = m->wsize;
    const int64_t head_stride = (int64_t)cap * c.head_dim;
    // one-row draft forwards read the draft's FP8 copy of a layer where it has one
    const bool fp8 = m->has_fp8 && skip && max_rows == 1;
    auto lin = [&](int kind, int l, const void *W, const float *X, int64_t ldx, const void *gain, const EpiArgs &e,
                   const uint16_t *xs) {
        if (fp8 && m->fp8_q[l][kind]) {
            Plan q = P[kind];
            q.path = PATH_GEMV_FP8;
            return run_linear(m, w, q, max_rows, m->fp8_q[l][kind], X, ldx, gain, e, xs, cur->guarded,
                              m->fp8_e[l][kind]);
        }
        return run_linear(m, w, P[kind], max_rows, W, X, ldx, gain, e, xs, cur->guarded);
    };
    for (int l = cur->next_layer; l < layer_end; ++l) {
        if (!(skip && skip[2 * l])) {
            char *kbase = static_cast<char *>(kv) + (size_t)(2 * l) * c.n_kv_heads * head_stride * ksz;
            char *vbase = static_cast<char *>(kv) + (size_t)(2 * l + 1) * c.n_kv_heads * head_stride * ksz;
            EpiArgs e{};
            e.q = w.q;
            e.ld_q = ldq;
            e.kcache = kbase;
            e.vcache = vbase;
            e.kv_head_stride = head_stride;
            e.rope = m->rope;
            e.n_heads = c.n_heads;
            e.n_kv_heads = c.n_kv_heads;
            e.head_dim = c.head_dim;
            e.ffn = c.ffn_dim;
            SD_TRY(prep_norm(m, w, P[LK_QKV], m->attn_norm[l], pending));
            SD_TRY(lin(LK_QKV, l, m->w_qkv[l], w.h, ldh, m->attn_norm[l], e, w.xa));
            AttnArgs at{};
            at.q = w.q;
            at.ld_q = ldq;
            at.kcache = kbase;
            at.vcache = vbase;
            at.kv_head_stride = head_stride;
            at.part_o = w.attn_o;
            at.part_ml = w.attn_ml;
            at.out = w.o;
            at.ld_out = ldq;
            if (P[LK_O].path == PATH_MFMA) {
                at.out_x = w.xa;
                at.ld_out = w.xld;
            }
            at.n_heads = c.n_heads;
            at.n_kv_heads = c.n_kv_heads;
            at.head_dim = c.head_dim;
            at.cap = cap;
            at.ctl = w.ctl;
            SD_TRY(launch(launch_attention(at, m->bf16, max_rows, m->stream), "attention"));
            EpiArgs eo{};
            eo.out = w.h;
            eo.ld_out = ldh;
            SD_TRY(lin(LK_O, l, m->w_o[l], w.o, ldq, nullptr, eo, w.xa));
            if (P[LK_O].epi == EPI_PARTIAL)
                pending = P[LK_O].splits;
        }
        if (!(skip && skip[2 * l + 1])) {
            EpiArgs eg{};
            eg.out = w.mbuf;
            eg.ld_out = c.ffn_dim;
            eg.ffn = c.ffn_dim;
            if (P[LK_DOWN].path == PATH_MFMA) {
                eg.out_x = w.xb;
                eg.ld_out = w.xld;
            }
            SD_TRY(prep_norm(m, w, P[LK_GATE_UP], m->mlp_norm[l], pending));
            SD_TRY(lin(LK_GATE_UP, l, m->w_gate_up[l], w.h, ldh, m->mlp_norm[l], eg, w.xa));
            EpiArgs ed{};
            ed.out = w.h;
            ed.ld_out = ldh;
            SD_TRY(lin(LK_DOWN, l, m->w_down[l], w.mbuf, c.ffn_dim, nullptr, ed, w.xb));
            if (P[LK_DOWN].epi == EPI_PARTIAL)
                pending = P[LK_DOWN].splits;
        }
    }
    cur->next_layer = std::max(cur->next_layer, layer_end);
    return SD_OK;
}

sd_status forward_head(sd_model *m, const Workspace &w, ForwardCursor *cur, const HeadSpec &hs) {
    if (!hs.run)
        return SD_OK;
    const sd_config &c = m->cfg;
    const Plan *P = cur->P;
    EpiArgs eh{};
    eh.head.mode = hs.mode;
    eh.head.logits = hs.logits;
    eh.head.ld_logits = c.vocab;
    eh.head.partials = w.head_part;
    eh.head.st = m->st;
    eh.head.mb = m->mb_dev;
    eh.head.out_tokens = m->d_out;
    eh.head.stage_log = m->d_log;
    eh.head.gamma_log = m->d_glog;
    eh.head.stage_log_cap = std::min(m->d_log_cap / 2, m->d_glog_cap);
    if (hs.sampled) {
        eh.head.sampled = 1;
        eh.head.logits = hs.mode == HEAD_DRAFT ? m->slog_d : m->slog_v;
        eh.head.logits_by_draft = hs.mode == HEAD_DRAFT;
    }
    SD_TRY(prep_norm(m, w, P[LK_HEAD], m->final_norm, cur->pending));
    return run_linear(m, w, P[LK_HEAD], cur->max_rows, m->lm_head, w.h, c.d_model, m->final_norm, eh, w.xa);
}

sd_status enqueue_forward(sd_model *m, const Workspace &w, void *kv, int32_t cap, const uint8_t *skip, int max_rows,
                          const HeadSpec &hs) {
    ForwardCursor cur;
    SD_TRY(forward_begin(m, w, max_rows, &cur));
    SD_TRY(forward_layers(m, w, kv, cap, skip, &cur, m->cfg.n_layers));
    return forward_head(m, w, &cur, hs);
}

size_t kv_bytes(const sd_config &c, int32_t cap) {
    const size_t es = c.dtype == SD_BF16 ? 2 : 4;
    return (size_t)c.n_layers * 2 * (size_t)c.n_kv_heads * (size_t)cap * (size_t)c.head_dim * es;
}

sd_status check_config(const sd_config *c) {
    if (!c)
        return fail(SD_ERR_INVALID_ARG, "config is null");
    if (c->n_layers < 1 || c->d_model < 8 || c->d_model % 8 || c->n_heads < 1 || c->n_kv_heads < 1 ||
        c->n_heads % c->n_kv_heads || c->head_dim < 16 || (c->head_dim & (c->head_dim - 1)) ||
        c->head_dim > MAX_HEAD_DIM ||
        c->ffn_dim < 8 || c->ffn_dim % 8 || c->vocab < 2 || (c->n_heads * c->head_dim) % 8)
        return fail(SD_ERR_INVALID_ARG, "unsupported model shape (need d_model and ffn_dim multiples of 8, head_dim "
                                        "a power of two in [16, 128], n_heads a multiple of n_kv_heads)");
    if (c->dtype != SD_F32 && c->dtype != SD_BF16)
        return fail(SD_ERR_INVALID_ARG, "dtype must be SD_F32 or SD_BF16");
    if (!(c->rms_eps > 0.0f) || !(c->rope_base > 0.0f))
        return fail(SD_ERR_INVALID_ARG, "rms_eps and rope_base must be positive");
    return SD_OK;
}

sd_status check_tokens(const sd_model *m, const int32_t *t, int32_t n, const char *what) {
    if (!t)
        return fail(SD_ERR_INVALID_ARG, std::string(what) + " is null");
    for (int32_t i = 0; i < n; ++i)
        if (t[i] < 0 || t[i] >= m->cfg.vocab)
            return fail(SD_ERR_INVALID_ARG, std::string(what) + "[" + std::to_string(i) + "] = " +
                                                std::to_string(t[i]) + " is outside [0, vocab)");
    return SD_OK;
}

sd_status check_mask(const sd_model *m, const uint8_t *skip) {
    if (!skip)
        return SD_OK;
    for (int i = 0; i < 2 * m->cfg.n_layers; ++i)
        if (skip[i] > 1)
            return fail(SD_ERR_INVALID_ARG, "skip_mask entries must be 0 or 1");
    return SD_OK;
}

sd_status create_cache(sd_model *m, int32_t cap, void *buf, sd_kv_cache **out) {
    if (cap < 1)
        return fail(SD_ERR_INVALID_ARG, "capacity must be >= 1");
    if (cap > MAX_CONTEXT)
        return fail(SD_ERR_CAPACITY, "capacity above " + std::to_string(MAX_CONTEXT) + " positions");
    if (buf && !aligned16(buf))
        return fail(SD_ERR_INVALID_ARG, "cache buffer must be 16-byte aligned");
    SD_TRY(ensure_rope(m, cap));
    SD_TRY(ensure_attn(m, cap));
    sd_kv_cache *c = new (std::nothrow) sd_kv_cache{m, buf, buf == nullptr, cap, 0};
    if (!c)
        return fail(SD_ERR_OOM, "host allocation failed");
    if (!buf) {
        if (hipMalloc(&c->buf, kv_bytes(m->cfg, cap)) != hipSuccess) {
            delete c;
            return fail(SD_ERR_OOM, "KV cache allocation of " + std::to_string(kv_bytes(m->cfg, cap)) +
                                        " bytes failed");
        }
    }
    *out = c;
    return SD_OK;
}

void destroy_cache(sd_kv_cache *c) {
    if (!c)
        return;
    if (c->owns)
        dev_free(c->buf);
    delete c;
}

// Caches the caller creates are registered with their model; destroying the
// model detaches them (model = nullptr) so that they can still be destroyed.
sd_status create_user_cache(sd_model *m, int32_t cap, void *buf, sd_kv_cache **out) {
    m->caches.reserve(m->caches.size() + 1);  // registration below cannot throw
    SD_TRY(create_cache(m, cap, buf, out));
    m->caches.push_back(*out);
    return SD_OK;
}

void destroy_user_cache(sd_kv_cache *c) {
    if (sd_model *m = c->model) {
        (void)hipStreamSynchronize(m->stream);
        auto it = std::find(m->caches.begin(), m->caches.end(), c);
        if (it != m->caches.end())
            m->caches.erase(it);
    }
    destroy_cache(c);
}

sd_status ensure_gen_cache(sd_model *m, int32_t cap) {
    if (m->gen_cache && m->gen_cache->cap >= cap)
        return SD_OK;
    SD_HIP(hipStreamSynchronize(m->stream));
    destroy_cache(m->gen_cache);
    m->gen_cache = nullptr;
    return create_cache(m, cap, nullptr, &m->gen_cache);
}

// Large-M forward (bfloat16 models): the M <= PF_ROWS tokens dev_tokens at
// positions [start, start + M), matrix-core GEMMs over all rows at once;
// logits (device [M][vocab]) when not null.
sd_status enqueue_forward_large(sd_model *m, void *kv, int32_t cap, const uint8_t *skip, const int32_t *dev_tokens,
                                int32_t M, int32_t start, float *logits) {
    const sd_config &c = m->cfg;
    const int H = c.n_heads, KVH = c.n_kv_heads, dh = c.head_dim, d = c.d_model, F = c.ffn_dim;
    const int hd = H * dh, nq = (H + 2 * KVH) * dh;
    const int64_t head_stride = (int64_t)cap * dh;
    const int64_t xt = m->pf_term;
    hipStream_t s = m->stream;
    // A split residual update leaves its partials in pf_part; the next norm
    // adds them into the residual stream (fold = their count, 0: none).
    int fold = 0;
    auto gemm = [&](const void *W, int N, int K, float *C, int64_t ldc, int epi, const uint16_t *A, int64_t a_term) {
        PfGemmArgs g{};
        g.W = static_cast<const uint16_t *>(W);
        g.A = A;
        g.a_term = a_term;
        g.C = C;
        g.ldc = ldc;
        g.M = M;
        g.N = N;
        g.K = K;
        g.lda = K;
        g.part = epi == EPI_RESID ? m->pf_part : nullptr;  // [PF_MAX_SPLITS][M][d]: split reductions
        // EPI_SWIGLU: the MLP activation terms, not into A (other work-groups
        // still read it)
        g.xout = m->pf_y;
        g.x_term = m->pf_y_term;
        return launch(launch_pf_gemm(g, epi, s, epi == EPI_RESID && C == m->pf_h ? &fold : nullptr), "prefill GEMM");
    };
    auto norm = [&](const void *gain) {
        const uint16_t *g = static_cast<const uint16_t *>(gain);
        if (fold) {
            const int f = fold;
            fold = 0;
            return launch(launch_pf_fold_norm_split(m->pf_h, m->pf_part, f, d, M, g, c.rms_eps, m->pf_x, xt, s),
                          "prefill norm");
        }
        return launch(launch_pf_norm_split(m->pf_h, d, M, g, c.rms_eps, m->pf_x, xt, s), "prefill norm");
    };
    SD_TRY(launch(launch_pf_embed(static_cast<const uint16_t *>(m->tok_emb), d, dev_tokens, M, m->pf_h, s),
                  "prefill embedding"));
    for (int l = 0; l < c.n_layers; ++l) {
        if (!(skip && skip[2 * l])) {
            uint16_t *kbase = reinterpret_cast<uint16_t *>(kv) + (size_t)(2 * l) * KVH * head_stride;
            uint16_t *vbase = reinterpret_cast<uint16_t *>(kv) + (size_t)(2 * l + 1) * KVH * head_stride;
            SD_TRY(norm(m->attn_norm[l]));
            SD_TRY(gemm(m->w_qkv[l], nq, d, m->pf_c, nq, EPI_STORE, m->pf_x, xt));
            SD_TRY(launch(launch_pf_rope_kv(m->pf_c, M, start, m->rope, H, KVH, dh, m->pf_q, kbase, vbase,
                                            head_stride, s),
                          "prefill rotary"));
            PfAttnArgs at{};
            at.q = m->pf_q;
            at.ldq = hd;
            at.kcache = kbase;
            at.vcache = vbase;
            at.kv_head_stride = head_stride;
            at.out = m->pf_x;
            at.out_term = xt;
            at.ldo = hd;
            at.M = M;
            at.start = start;
            at.n_heads = H;
            at.n_kv_heads = KVH;
            at.head_dim = dh;
            SD_TRY(launch(launch_pf_attention(at, s), "prefill attention"));
            SD_TRY(gemm(m->w_o[l], d, hd, m->pf_h, d, EPI_RESID, m->pf_x, xt));
        }
        if (!(skip && skip[2 * l + 1])) {
            SD_TRY(norm(m->mlp_norm[l]));
            SD_TRY(gemm(m->w_gate_up[l], 2 * F, d, m->pf_c, 2 * F, EPI_SWIGLU, m->pf_x, xt));
            SD_TRY(gemm(m->w_down[l], d, F, m->pf_h, d, EPI_RESID, m->pf_y, m->pf_y_term));
        }
    }
    if (logits) {
        SD_TRY(norm(m->final_norm));
        SD_TRY(gemm(m->lm_head, c.vocab, d, logits, c.vocab, EPI_STORE, m->pf_x, xt));
    } else if (fold) {
        // no norm follows: leave the residual stream whole
        SD_TRY(launch(launch_pf_split_sum(m->pf_part, fold, (int64_t)M * d, m->pf_h, s), "prefill split sum"));
    }
    return SD_OK;
}

// Prefill: full-model forward of tokens [0, n) already on the device, no
// head: PF_ROWS-row chunks on the large-M path (bfloat16 models, more than
// MAX_ROWS tokens), else MAX_ROWS-row chunks.
sd_status enqueue_prefill(sd_model *m, sd_kv_cache *kc, const int32_t *dev_tokens, int32_t n, int32_t start) {
    if (m->pf_ok && n > MAX_ROWS) {
        for (int32_t c = 0; c < n; c += PF_ROWS)
            SD_TRY(enqueue_forward_large(m, kc->buf, kc->cap, nullptr, dev_tokens + c, std::min(PF_ROWS, n - c),
                                         start + c, nullptr));
        return SD_OK;
    }
    for (int32_t c = 0; c < n; c += MAX_ROWS) {
        const int32_t rows = std::min<int32_t>(MAX_ROWS, n - c);
        SD_TRY(launch(launch_set_ctl(m->ws.ctl, start + c, rows, dev_tokens + c, m->stream), "control block"));
        SD_TRY(enqueue_forward(m, m->ws, kc->buf, kc->cap, nullptr, rows, HeadSpec{}));
    }
    return SD_OK;
}

// Waits until the mailbox shows step seq; *word receives what it holds.
sd_status wait_mailbox(sd_model *m, int32_t seq, uint64_t *word) {
    uint64_t spins = 0;
    for (;;) {
        const uint64_t w = __atomic_load_n(&m->mb_host->word, __ATOMIC_ACQUIRE);
        if (mb_seq(w) == seq) {
            *word = w;
            return SD_OK;
        }
        if ((++spins & 1023u) == 0) {
            const hipError_t e = hipStreamQuery(m->stream);
            if (e == hipSuccess) {
                const uint64_t w2 = __atomic_load_n(&m->mb_host->word, __ATOMIC_ACQUIRE);
                if (mb_seq(w2) == seq) {
                    *word = w2;
                    return SD_OK;
                }
                return fail(SD_ERR_DEVICE, "decode step " + std::to_string(seq) +
                                               " finished without posting its result");
            }
            if (e != hipErrorNotReady)
                return fail(SD_ERR_DEVICE, std::string("decode step failed: ") + hipGetErrorString(e));
        }
#if defined(__x86_64__)
        _mm_pause();
#endif
    }
}

float elapsed(hipEvent_t a, hipEvent_t b);

// Adds up the timed launches of the finished call (the stream is idle).
void collect_timing(sd_model *m) {
    for (size_t i = 0; i + 1 < m->tev_used; i += 2) {
        m->timed_ms += elapsed(m->tev[i], m->tev[i + 1]);
        m->timed_launches += 1;
    }
    m->tev_used = 0;
}

float elapsed(hipEvent_t a, hipEvent_t b) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess)
        return 0.0f;
    return ms;
}

sd_status copy_results(sd_model *m, int32_t max_new, int32_t *out_tokens, sd_stats *stats) {
    if (max_new > 0)
        SD_HIP(hipMemcpyAsync(out_tokens, m->d_out, sizeof(int32_t) * (size_t)max_new, hipMemcpyDeviceToHost,
                              m->stream));
    DevState st{};
    SD_HIP(hipMemcpyAsync(&st, m->st, sizeof st, hipMemcpyDeviceToHost, m->stream));
    std::vector<int32_t> log;
    std::vector<float> glog;
    int64_t nlog = 0;
    if (stats && (stats->stage_log || stats->gamma_log) && stats->stage_log_cap > 0) {
        nlog = std::min<int64_t>(stats->stage_log_cap, std::min(m->d_log_cap / 2, m->d_glog_cap));
        log.resize((size_t)nlog * 2);
        glog.resize((size_t)nlog);
        SD_HIP(hipMemcpyAsync(log.data(), m->d_log, sizeof(int32_t) * 2 * (size_t)nlog, hipMemcpyDeviceToHost,
                              m->stream));
        SD_HIP(hipMemcpyAsync(glog.data(), m->d_glog, sizeof(float) * (size_t)nlog, hipMemcpyDeviceToHost,
                              m->stream));
    }
    SD_HIP(hipStreamSynchronize(m->stream));
    collect_timing(m);
    if (stats) {
        stats->n_stages = st.n_stages;
        stats->n_drafted = st.n_drafted;
        stats->n_accepted = st.n_accepted;
        stats->n_emitted = st.emitted;
        stats->n_draft_steps = st.n_draft_steps;
        if (nlog) {
            const int64_t n = std::min<int64_t>(nlog, st.n_stages);
            if (stats->stage_log)
                std::memcpy(stats->stage_log, log.data(), sizeof(int32_t) * 2 * (size_t)n);
            if (stats->gamma_log)
                std::memcpy(stats->gamma_log, glog.data(), sizeof(float) * (size_t)n);
        }
    }
    return SD_OK;
}

sd_status check_generate(sd_model *m, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                         int32_t *out_tokens) {
    if (!m)
        return fail(SD_ERR_INVALID_ARG, "model is null");
    if (prompt_len < 1)
        return fail(SD_ERR_INVALID_ARG, "prompt_len must be >= 1");
    if (max_new < 0)
        return fail(SD_ERR_INVALID_ARG, "max_new must be >= 0");
    if (max_new > 0 && !out_tokens)
        return fail(SD_ERR_INVALID_ARG, "out_tokens is null");
    if ((int64_t)prompt_len + max_new + MAX_ROWS > (int64_t)INT32_MAX / 2)
        return fail(SD_ERR_INVALID_ARG, "prompt_len + max_new too large");
    return check_tokens(m, prompt, prompt_len, "prompt");
}

// Shared start of both generate calls: buffers, prompt upload, prefill,
// decode-state setup.
sd_status start_generate(sd_model *m, const int32_t *prompt, int32_t prompt_len, int32_t max_new, int32_t k_max,
                         const ExitRule &rule) {
    SD_TRY(ensure_gen_cache(m, prompt_len + max_new + k_max + 1));
    SD_TRY(ensure_buf(m, &m->d_tokens, &m->d_tokens_cap, prompt_len));
    SD_TRY(ensure_buf(m, &m->d_out, &m->d_out_cap, std::max(max_new, 1)));
    SD_TRY(ensure_buf(m, &m->d_log, &m->d_log_cap, 2 * std::max(max_new, 1)));
    SD_TRY(ensure_buf(m, &m->d_glog, &m->d_glog_cap, std::max(max_new, 1)));
    SD_HIP(hipMemcpyAsync(m->d_tokens, prompt, sizeof(int32_t) * (size_t)prompt_len, hipMemcpyHostToDevice,
                          m->stream));
    SD_HIP(hipEventRecord(m->ev[0], m->stream));
    m->gen_cache->len = 0;
    SD_TRY(enqueue_prefill(m, m->gen_cache, m->d_tokens, prompt_len - 1, 0));
    m->gen_cache->len = prompt_len - 1;
    SD_HIP(hipEventRecord(m->ev[1], m->stream));
    __atomic_store_n(&m->mb_host->word, mb_pack(-1, 0, 0, 0), __ATOMIC_RELEASE);
    SD_TRY(launch(launch_init_decode(m->st, m->ws.ctl, m->mb_dev, prompt_len - 1, m->d_tokens + prompt_len - 1,
                                     max_new, k_max, rule, m->stream),
                  "decode setup"));
    return SD_OK;
}

// Checks and installs the parameters of the sampling variant (sp == null:
// greedy decoding).
sd_status use_sampling(sd_model *m, const SampleParams *sp) {
    if (!sp)
        return SD_OK;
    if (!(sp->temperature > 0.0f) || !std::isfinite(sp->temperature))
        return fail(SD_ERR_INVALID_ARG, "temperature must be positive and finite");
    if (!(sp->top_p > 0.0f) || !(sp->top_p <= 1.0f))
        return fail(SD_ERR_INVALID_ARG, "top_p must be in (0, 1]");
    if (m->cfg.vocab > MAX_SAMPLE_VOCAB)
        return fail(SD_ERR_INVALID_ARG, "sampling takes vocabularies of at most 524288 ids");
    m->sp_cur = *sp;
    return SD_OK;
}

sd_status self_spec(sd_model *m, const int32_t *prompt, int32_t prompt_len, int32_t max_new, const uint8_t *skip,
                    int32_t k_max, const ExitRule &rule, const SampleParams *sp, int32_t *out_tokens,
                    sd_stats *stats) {
    SD_TRY(check_generate(m, prompt, prompt_len, max_new, out_tokens));
    if (k_max < 0 || k_max > MAX_ROWS - 1)
        return fail(SD_ERR_INVALID_ARG, "K_max must be in [0, 15]");
    if (std::isnan(rule.gamma))
        return fail(SD_ERR_INVALID_ARG, "gamma is NaN");
    if (rule.adaptive && (std::isnan(rule.gamma0) || std::isnan(rule.alpha) || std::isnan(rule.epsilon) ||
                          std::isnan(rule.beta1) || std::isnan(rule.beta2)))
        return fail(SD_ERR_INVALID_ARG, "adaptive parameters must not be NaN");
    SD_TRY(check_mask(m, skip));
    SD_TRY(use_sampling(m, sp));
    SD_TRY(start_generate(m, prompt, prompt_len, max_new, k_max, rule));
    sd_kv_cache *kc = m->gen_cache;
    const Workspace &w = m->ws;
    const int L = m->cfg.n_layers;

    // The device decides every step (draft or verification, and how many
    // rows) and posts the decision to the pinned mailbox.  So that the GPU
    // never waits for the host, the host keeps the first part of the next
    // step enqueued ahead on a prediction while it waits for the current
    // step's decision: a guard kernel, the embedding and the layers up to
    // the step's first sublayer.  If the decision asks for another step,
    // the guard has cancelled the part (every kernel sees zero rows and
    // writes nothing) and the host enqueues the right step in full.
    struct Step {
        int phase, rows;
    };
    auto split_layer = [&](const uint8_t *sk) {
        int run = 0;
        for (int l = 0; l < L; ++l) {
            run += (sk && sk[2 * l] ? 0 : 1) + (sk && sk[2 * l + 1] ? 0 : 1);
            if (run >= 1)
                return l + 1;
        }
        return L;
    };
    const int split_draft = split_layer(skip), split_verify = split_layer(nullptr);

    // GPU time per slot: each enqueued step, or cancelled part, is bracketed
    // by two events from a ring; a slot is read once it has surely finished.
    struct Slot {
        int kind;  // PHASE_DRAFT, PHASE_VERIFY, or -1: cancelled
        hipEvent_t a, b;
    };
    std::vector<Slot> open_slots;
    int ring = 0;
    double draft_ms = 0.0, verify_ms = 0.0, noop_ms = 0.0;
    int64_t n_noop = 0;
    hipEvent_t last_end = nullptr;
    auto slot_open = [&]() -> sd_status {
        Slot sl{-2, m->ev[2 + 2 * ring], m->ev[3 + 2 * ring]};
        ring = (ring + 1) % STEP_EVENT_PAIRS;
        SD_HIP(hipEventRecord(sl.a, m->stream));
        open_slots.push_back(sl);
        return SD_OK;
    };
    auto slot_close = [&](int kind) -> sd_status {
        Slot &sl = open_slots.back();
        sl.kind = kind;
        SD_HIP(hipEventRecord(sl.b, m->stream));
        last_end = sl.b;
        return SD_OK;
    };
    auto account = [&](size_t keep) {  // all but the last `keep` slots have finished
        size_t n = open_slots.size() > keep ? open_slots.size() - keep : 0;
        for (size_t i = 0; i < n; ++i) {
            const Slot &sl = open_slots[i];
            const float ms = elapsed(sl.a, sl.b);
            (sl.kind == PHASE_DRAFT ? draft_ms : sl.kind == PHASE_VERIFY ? verify_ms : noop_ms) += ms;
        }
        open_slots.erase(open_slots.begin(), open_slots.begin() + (ptrdiff_t)n);
    };
    auto begin_step = [&](const Step &st, ForwardCursor *cur) -> sd_status {
        SD_TRY(slot_open());
        SD_TRY(launch(launch_step_guard(w.ctl, m->st, st.phase, st.rows, m->stream), "step guard"));
        SD_TRY(forward_begin(m, w, st.rows, cur));
        cur->guarded = true;
        return forward_layers(m, w, kc->buf, kc->cap, st.phase == PHASE_DRAFT ? skip : nullptr, cur,
                              st.phase == PHASE_DRAFT ? split_draft : split_verify);
    };
    auto finish_step = [&](const Step &st, ForwardCursor *cur) -> sd_status {
        cur->guarded = false;  // the host has seen the decision: the step runs
        SD_TRY(forward_layers(m, w, kc->buf, kc->cap, st.phase == PHASE_DRAFT ? skip : nullptr, cur, L));
        HeadSpec hs;
        hs.run = true;
        hs.sampled = sp != nullptr;
        hs.mode = st.phase == PHASE_DRAFT ? HEAD_DRAFT : HEAD_VERIFY;
        SD_TRY(forward_head(m, w, cur, hs));
        return slot_close(st.phase);
    };

    // The host mirrors the stage: drafts enqueued in it, the draft budget
    // (from the tokens emitted before it), and the previous stage's length,
    // which predicts where this one ends.
    int stage_k = 0, prev_stage_k = 1;
    int kcap = std::min(k_max, max_new - 1);
    auto apply = [&](const Step &st) {
        if (st.phase == PHASE_DRAFT) {
            ++stage_k;
        } else {
            prev_stage_k = std::max(stage_k, 1);
            stage_k = 0;
        }
    };
    auto predict = [&](const Step &prev) -> Step {
        if (prev.phase == PHASE_DRAFT && (stage_k >= kcap || stage_k >= prev_stage_k))
            return Step{PHASE_VERIFY, stage_k + 1};
        return Step{PHASE_DRAFT, 1};
    };
    if (max_new > 0) {
        Step cur_step{kcap > 0 ? PHASE_DRAFT : PHASE_VERIFY, 1};
        ForwardCursor cur, ahead;
        SD_TRY(begin_step(cur_step, &cur));
        SD_TRY(finish_step(cur_step, &cur));
        apply(cur_step);
        int32_t seq = 1;
        Step pred = predict(cur_step);
        size_t tev_mark = m->tev_used;
        SD_TRY(begin_step(pred, &ahead));
        for (;;) {
            uint64_t word = 0;
            SD_TRY(wait_mailbox(m, seq, &word));
            account(2);  // the current step's end event and the part ahead may still be pending
            if (cur_step.phase == PHASE_VERIFY)
                kcap = std::min(k_max, max_new - mb_emitted(word) - 1);
            const bool done = mb_done(word);
            const Step truth{mb_phase(word), mb_phase(word) == PHASE_DRAFT ? 1 : stage_k + 1};
            if (!done && truth.phase == pred.phase && truth.rows == pred.rows) {
                SD_TRY(finish_step(pred, &ahead));
            } else {
                // cancelled on the device by its guard; its timed launches
                // (measurement hook) are dropped
                SD_TRY(slot_close(-1));
                m->tev_used = tev_mark;
                ++n_noop;
                if (done)
                    break;
                SD_TRY(begin_step(truth, &cur));
                SD_TRY(finish_step(truth, &cur));
            }
            cur_step = truth;
            apply(cur_step);
            ++seq;
            pred = predict(cur_step);
            tev_mark = m->tev_used;
            SD_TRY(begin_step(pred, &ahead));
        }
    }
    SD_TRY(copy_results(m, max_new, out_tokens, stats));
    account(0);
    if (stats) {
        stats->draft_ms = draft_ms;
        stats->verify_ms = verify_ms;
        stats->noop_ms = noop_ms;
        stats->n_guarded_noop_steps = n_noop;
        stats->prefill_ms = elapsed(m->ev[0], m->ev[1]);
        stats->total_ms = last_end ? elapsed(m->ev[0], last_end) : stats->prefill_ms;
        stats->decode_ms = stats->total_ms - stats->prefill_ms;
    }
    kc->len = 0;
    return SD_OK;
}

sd_status autoregressive(sd_model *m, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                         const SampleParams *sp, int32_t *out_tokens, sd_stats *stats) {
    SD_TRY(check_generate(m, prompt, prompt_len, max_new, out_tokens));
    SD_TRY(use_sampling(m, sp));
    SD_TRY(start_generate(m, prompt, prompt_len, max_new, 0, ExitRule{}));
    sd_kv_cache *kc = m->gen_cache;
    HeadSpec hs;
    hs.run = true;
    hs.mode = HEAD_AR;
    hs.sampled = sp != nullptr;
    for (int32_t i = 0; i < max_new; ++i)
        SD_TRY(enqueue_forward(m, m->ws, kc->buf, kc->cap, nullptr, 1, hs));
    SD_HIP(hipEventRecord(m->ev[2], m->stream));
    SD_TRY(copy_results(m, max_new, out_tokens, stats));
    if (stats) {
        stats->prefill_ms = elapsed(m->ev[0], m->ev[1]);
        stats->total_ms = elapsed(m->ev[0], m->ev[2]);
        stats->decode_ms = stats->total_ms - stats->prefill_ms;
        stats->draft_ms = 0.0;
        stats->verify_ms = stats->decode_ms;
        stats->n_stages = 0;
        stats->n_guarded_noop_steps = 0;
        stats->noop_ms = 0.0;
    }
    kc->len = 0;
    return SD_OK;
}

sd_status forward(sd_model *m, const int32_t *tokens, int32_t n, const uint8_t *skip, sd_kv_cache *kc,
                  float *logits) {
    if (!m || !kc)
        return fail(SD_ERR_INVALID_ARG, "model or cache is null");
    if (kc->model != m)
        return fail(SD_ERR_INVALID_ARG, "cache belongs to another model");
    if (n < 1)
        return fail(SD_ERR_INVALID_ARG, "n must be >= 1");
    SD_TRY(check_tokens(m, tokens, n, "tokens"));
    SD_TRY(check_mask(m, skip));
    if (skip && n > 1 && m->has_fp8)
        return fail(SD_ERR_INVALID_ARG, "while the draft is quantized, forwards with a skip mask take one row");
    if ((int64_t)kc->len + n > kc->cap)
        return fail(SD_ERR_CAPACITY, "cache of capacity " + std::to_string(kc->cap) + " holds " +
                                         std::to_string(kc->len) + " positions; " + std::to_string(n) +
                                         " more do not fit");
    SD_TRY(ensure_buf(m, &m->d_tokens, &m->d_tokens_cap, n));
    SD_HIP(hipMemcpyAsync(m->d_tokens, tokens, sizeof(int32_t) * (size_t)n, hipMemcpyHostToDevice, m->stream));
    for (int32_t c = 0; m->pf_ok && n > MAX_ROWS && c < n; c += PF_ROWS)
        SD_TRY(enqueue_forward_large(m, kc->buf, kc->cap, skip, m->d_tokens + c, std::min(PF_ROWS, n - c),
                                     kc->len + c, logits ? logits + (size_t)c * m->cfg.vocab : nullptr));
    for (int32_t c = 0; !(m->pf_ok && n > MAX_ROWS) && c < n; c += MAX_ROWS) {
        const int32_t rows = std::min<int32_t>(MAX_ROWS, n - c);
        SD_TRY(launch(launch_set_ctl(m->ws.ctl, kc->len + c, rows, m->d_tokens + c, m->stream), "control block"));
        HeadSpec hs;
        hs.run = logits != nullptr;
        hs.mode = HEAD_NONE;
        hs.logits = logits ? logits + (size_t)c * m->cfg.vocab : nullptr;
        SD_TRY(enqueue_forward(m, m->ws, kc->buf, kc->cap, skip, rows, hs));
    }
    SD_HIP(hipStreamSynchronize(m->stream));
    collect_timing(m);
    kc->len += n;
    return SD_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// Allocation-free forward (sd_forward_static).  Its scratch lives in this
// file-scope device array: each GPU the library runs on holds its own copy
// until the process ends.  Host code never passes the array's name to a
// kernel (on the host it only names a stand-in): the device address comes
// from hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t STATIC_SCRATCH_BYTES = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

namespace {

constexpr int MAX_SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
char *g_scratch[MAX_SCRATCH_DEVICES] = {};

// Device address of the scratch array on the device of stream s.
sd_status scratch_base(hipStream_t s, char **out) {
    int cur = -1;
    SD_HIP(hipGetDevice(&cur));
    int dev = cur;
    if (s)
        SD_HIP(hipStreamGetDevice(s, &dev));
    if (dev < 0 || dev >= MAX_SCRATCH_DEVICES)
        return fail(SD_ERR_DEVICE, "device index " + std::to_string(dev) + " out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        if (dev != cur)
            SD_HIP(hipSetDevice(dev));
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur)
            (void)hipSetDevice(cur);
        if (e != hipSuccess || !p)
            return fail(SD_ERR_DEVICE, std::string("scratch address: ") + hipGetErrorString(e));
        g_scratch[dev] = static_cast<char *>(p);
    }
    *out = g_scratch[dev];
    return SD_OK;
}

// Lays out a forward's scratch for model m over a cache of capacity cap at
// base (or only sizes it when base is null); returns the bytes used.  Every
// buffer starts on a 256-byte boundary.
size_t carve_workspace(const sd_model *m, int32_t cap, char *base, Workspace *w) {
    const sd_config &c = m->cfg;
    size_t off = 0;
    auto take = [&](size_t bytes) -> char * {
        char *p = base ? base + off : nullptr;
        off += (bytes + 255) & ~(size_t)255;
        return p;
    };
    const size_t hd = (size_t)c.n_heads * c.head_dim, splits = (size_t)attn_split_slots(cap, attn_chunk_min_of(m));
    w->xld = xld_of(c);
    w->h = reinterpret_cast<float *>(take(sizeof(float) * MAX_ROWS * c.d_model));
    w->q = reinterpret_cast<float *>(take(sizeof(float) * MAX_ROWS * hd));
    w->o = reinterpret_cast<float *>(take(sizeof(float) * MAX_ROWS * hd));
    w->mbuf = reinterpret_cast<float *>(take(sizeof(float) * MAX_ROWS * c.ffn_dim));
    w->part = reinterpret_cast<float *>(take(sizeof(float) * 8 * MAX_ROWS * c.d_model));
    w->ssq = reinterpret_cast<float *>(take(sizeof(float) * MAX_ROWS * prep_slices(c.d_model)));
    w->xa = reinterpret_cast<uint16_t *>(take(sizeof(uint16_t) * X_TERMS * MAX_ROWS * w->xld));
    w->xb = reinterpret_cast<uint16_t *>(take(sizeof(uint16_t) * X_TERMS * MAX_ROWS * w->xld));
    w->head_part = reinterpret_cast<float4 *>(take(sizeof(float4) * m->max_head_tiles * MAX_ROWS));
    w->attn_o = reinterpret_cast<float *>(take(sizeof(float) * splits * c.n_heads * MAX_ROWS * c.head_dim));
    w->attn_ml = reinterpret_cast<float2 *>(take(sizeof(float2) * splits * c.n_heads * MAX_ROWS));
    w->ctl = reinterpret_cast<DevCtl *>(take(sizeof(DevCtl)));
    return off;
}

sd_status forward_static(sd_model *m, const int32_t *tokens, int32_t n, const uint8_t *skip, sd_kv_cache *kc,
                         float *logits) {
    if (!m || !kc)
        return fail(SD_ERR_INVALID_ARG, "model or cache is null");
    if (kc->model != m)
        return fail(SD_ERR_INVALID_ARG, "cache belongs to another model");
    if (n < 1 || n > MAX_ROWS)
        return fail(SD_ERR_INVALID_ARG, "n must be in [1, " + std::to_string(MAX_ROWS) + "]");
    SD_TRY(check_tokens(m, tokens, n, "tokens"));
    SD_TRY(check_mask(m, skip));
    if (skip && n > 1 && m->has_fp8)
        return fail(SD_ERR_INVALID_ARG, "while the draft is quantized, forwards with a skip mask take one row");
    if ((int64_t)kc->len + n > kc->cap)
        return fail(SD_ERR_CAPACITY, "cache of capacity " + std::to_string(kc->cap) + " holds " +
                                         std::to_string(kc->len) + " positions; " + std::to_string(n) +
                                         " more do not fit");
    Workspace w;
    const size_t need = carve_workspace(m, kc->cap, nullptr, &w);
    if (need > STATIC_SCRATCH_BYTES)
        return fail(SD_ERR_CAPACITY, "this model over a cache of " + std::to_string(kc->cap) + " positions needs " +
                                         std::to_string(need) + " bytes of scratch; the static array holds " +
                                         std::to_string(STATIC_SCRATCH_BYTES));
    char *base = nullptr;
    SD_TRY(scratch_base(m->stream, &base));
    carve_workspace(m, kc->cap, base, &w);
    // The array keeps the previous call's contents: the activation rows
    // start at zero, as a model's own workspace does.
    SD_TRY(launch(launch_fill_zero(w.h, sizeof(float) * MAX_ROWS * m->cfg.d_model, m->stream), "scratch clear"));
    SD_TRY(launch(launch_fill_zero(w.o, sizeof(float) * MAX_ROWS * m->cfg.n_heads * m->cfg.head_dim, m->stream),
                  "scratch clear"));
    SD_TRY(launch(launch_fill_zero(w.mbuf, sizeof(float) * MAX_ROWS * m->cfg.ffn_dim, m->stream), "scratch clear"));
    SD_TRY(launch(launch_set_ctl_host(w.ctl, kc->len, n, tokens, m->stream), "control block"));
    HeadSpec hs;
    hs.run = logits != nullptr;
    hs.mode = HEAD_NONE;
    hs.logits = logits;
    // the measurement hook's events stay out of this path
    const int timed = m->timed_kind;
    m->timed_kind = -1;
    const sd_status st = enqueue_forward(m, w, kc->buf, kc->cap, skip, n, hs);
    m->timed_kind = timed;
    SD_TRY(st);
    SD_HIP(hipStreamSynchronize(m->stream));
    kc->len += n;
    return SD_OK;
}

void free_draft_fp8(sd_model *m) {
    for (auto &a : m->fp8_q)
        for (uint8_t *&p : a) {
            dev_free(p);
            p = nullptr;
        }
    for (auto &a : m->fp8_e)
        for (int32_t *&p : a) {
            dev_free(p);
            p = nullptr;
        }
    m->has_fp8 = false;
}

// FP8 copies of the weights of the sublayers skip keeps (see k_quantize_fp8).
sd_status quantize_draft(sd_model *m, const uint8_t *skip) {
    if (!m)
        return fail(SD_ERR_INVALID_ARG, "model is null");
    SD_TRY(check_mask(m, skip));
    if (skip && !m->bf16)
        return fail(SD_ERR_INVALID_ARG, "FP8 draft weights are made from bfloat16 weights");
    const sd_config &c = m->cfg;
    if (skip && (c.d_model % 16 || (c.n_heads * c.head_dim) % 16 || c.ffn_dim % 16))
        return fail(SD_ERR_INVALID_ARG, "FP8 draft weights need d_model, n_heads * head_dim and ffn_dim multiples of 16");
    SD_HIP(hipStreamSynchronize(m->stream));
    free_draft_fp8(m);
    if (!skip)
        return SD_OK;
    const int L = c.n_layers;
    const int32_t rows[4] = {(c.n_heads + 2 * c.n_kv_heads) * c.head_dim, c.d_model, 2 * c.ffn_dim, c.d_model};
    const int32_t cols[4] = {c.d_model, c.n_heads * c.head_dim, c.d_model, c.ffn_dim};
    for (int l = 0; l < L; ++l) {
        const void *W[4] = {m->w_qkv[l], m->w_o[l], m->w_gate_up[l], m->w_down[l]};
        for (int k = 0; k < 4; ++k) {
            if (skip[2 * l + (k < LK_GATE_UP ? 0 : 1)])
                continue;
            sd_status st = dev_alloc(&m->fp8_q[l][k], (size_t)rows[k] * cols[k]);
            if (st == SD_OK)
                st = dev_alloc(&m->fp8_e[l][k], (size_t)rows[k]);
            if (st == SD_OK)
                st = launch(launch_quantize_fp8(static_cast<const uint16_t *>(W[k]), rows[k], cols[k], m->fp8_q[l][k],
                                                m->fp8_e[l][k], m->stream),
                            "FP8 quantization");
            if (st != SD_OK) {
                (void)hipStreamSynchronize(m->stream);
                free_draft_fp8(m);
                return st;
            }
            m->has_fp8 = true;
        }
    }
    const hipError_t e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) {
        free_draft_fp8(m);
        return fail(SD_ERR_DEVICE, std::string("FP8 quantization: ") + hipGetErrorString(e));
    }
    return SD_OK;
}

void destroy_model(sd_model *m) {
    if (!m)
        return;
    if (m->stream)
        (void)hipStreamSynchronize(m->stream);
    for (sd_kv_cache *c : m->caches)
        c->model = nullptr;
    free_draft_fp8(m);
    destroy_cache(m->gen_cache);
    dev_free(m->ws.h);
    dev_free(m->ws.q);
    dev_free(m->ws.o);
    dev_free(m->ws.mbuf);
    dev_free(m->ws.part);
    dev_free(m->ws.ssq);
    dev_free(m->ws.xa);
    dev_free(m->ws.xb);
    dev_free(m->ws.head_part);
    dev_free(m->slog_v);
    dev_free(m->slog_d);
    dev_free(m->svstat);
    dev_free(m->sdstat);
    dev_free(m->ws.attn_o);
    dev_free(m->ws.attn_ml);
    dev_free(m->rope);
    dev_free(m->pf_h);
    dev_free(m->pf_c);
    dev_free(m->pf_q);
    dev_free(m->pf_part);
    dev_free(m->pf_x);
    dev_free(m->pf_y);
    dev_free(m->ws.ctl);
    dev_free(m->st);
    dev_free(m->d_tokens);
    dev_free(m->d_out);
    dev_free(m->d_log);
    dev_free(m->d_glog);
    if (m->mb_host)
        (void)hipHostFree(m->mb_host);
    for (hipEvent_t &e : m->ev)
        if (e)
            (void)hipEventDestroy(e);
    for (hipEvent_t e : m->tev)
        (void)hipEventDestroy(e);
    delete m;
}

sd_status create_model(const sd_config *cfg, const sd_weights *w, void *stream, sd_model **out) {
    if (!out)
        return fail(SD_ERR_INVALID_ARG, "out is null");
    *out = nullptr;
    SD_TRY(check_config(cfg));
    if (!w)
        return fail(SD_ERR_INVALID_ARG, "weights is null");
    const int L = cfg->n_layers;
    auto ok = [](const void *p) { return p != nullptr && aligned16(p); };
    if (!ok(w->tok_emb) || !ok(w->final_norm) || !ok(w->lm_head) || !w->attn_norm || !w->w_qkv || !w->w_o ||
        !w->mlp_norm || !w->w_gate_up || !w->w_down)
        return fail(SD_ERR_INVALID_ARG, "a weight pointer is null or not 16-byte aligned");
    for (int l = 0; l < L; ++l)
        if (!ok(w->attn_norm[l]) || !ok(w->w_qkv[l]) || !ok(w->w_o[l]) || !ok(w->mlp_norm[l]) ||
            !ok(w->w_gate_up[l]) || !ok(w->w_down[l]))
            return fail(SD_ERR_INVALID_ARG, "a layer weight pointer is null or not 16-byte aligned (layer " +
                                                std::to_string(l) + ")");
    sd_model *m = new (std::nothrow) sd_model;
    if (!m)
        return fail(SD_ERR_OOM, "host allocation failed");
    m->cfg = *cfg;
    m->bf16 = cfg->dtype == SD_BF16;
    m->wsize = m->bf16 ? 2 : 4;
    m->tok_emb = w->tok_emb;
    m->final_norm = w->final_norm;
    m->lm_head = w->lm_head;
    m->attn_norm.assign(w->attn_norm, w->attn_norm + L);
    m->w_qkv.assign(w->w_qkv, w->w_qkv + L);
    m->w_o.assign(w->w_o, w->w_o + L);
    m->mlp_norm.assign(w->mlp_norm, w->mlp_norm + L);
    m->w_gate_up.assign(w->w_gate_up, w->w_gate_up + L);
    m->w_down.assign(w->w_down, w->w_down + L);
    m->fp8_q.assign(L, {nullptr, nullptr, nullptr, nullptr});
    m->fp8_e.assign(L, {nullptr, nullptr, nullptr, nullptr});
    m->stream = reinterpret_cast<hipStream_t>(stream);

    int max_head_tiles = 1;
    for (int k = 0; k < LK_COUNT; ++k) {
        m->plan1[k] = make_plan(m, (LinearKind)k, 1);
        m->plan2[k] = make_plan(m, (LinearKind)k, 2);
        m->planm[k] = make_plan(m, (LinearKind)k, 16);
        for (const Plan *p : {&m->plan1[k], &m->plan2[k], &m->planm[k]}) {
            if (k == LK_HEAD)
                max_head_tiles = std::max(max_head_tiles, head_tiles(*p));
        }
    }
    const sd_config &c = *cfg;
    sd_status st = SD_OK;
    auto chain = [&](sd_status s) {
        if (st == SD_OK)
            st = s;
    };
    Workspace &ws = m->ws;
    m->max_head_tiles = max_head_tiles;
    chain(dev_alloc(&ws.h, (size_t)MAX_ROWS * c.d_model));
    chain(dev_alloc(&ws.q, (size_t)MAX_ROWS * c.n_heads * c.head_dim));
    chain(dev_alloc(&ws.o, (size_t)MAX_ROWS * c.n_heads * c.head_dim));
    chain(dev_alloc(&ws.mbuf, (size_t)MAX_ROWS * c.ffn_dim));
    chain(dev_alloc(&ws.part, (size_t)8 * MAX_ROWS * c.d_model));
    chain(dev_alloc(&ws.ssq, (size_t)MAX_ROWS * prep_slices(c.d_model)));
    ws.xld = xld_of(c);
    chain(dev_alloc(&ws.xa, (size_t)X_TERMS * MAX_ROWS * ws.xld));
    chain(dev_alloc(&ws.xb, (size_t)X_TERMS * MAX_ROWS * ws.xld));
    chain(dev_alloc(&ws.head_part, (size_t)max_head_tiles * MAX_ROWS));
    chain(dev_alloc(&m->slog_v, (size_t)MAX_ROWS * c.vocab));
    chain(dev_alloc(&m->slog_d, (size_t)MAX_ROWS * c.vocab));
    chain(dev_alloc(&m->svstat, (size_t)MAX_ROWS));
    chain(dev_alloc(&m->sdstat, (size_t)MAX_ROWS));
    chain(dev_alloc(&ws.ctl, 1));
    chain(dev_alloc(&m->st, 1));
    m->pf_ok = m->bf16 && (c.head_dim == 32 || c.head_dim == 64 || c.head_dim == 128);
    if (m->pf_ok) {
        const int64_t hd = (int64_t)c.n_heads * c.head_dim;
        const int64_t nc = std::max<int64_t>((int64_t)(c.n_heads + 2 * c.n_kv_heads) * c.head_dim, 2 * c.ffn_dim);
        m->pf_term = (int64_t)PF_ROWS * std::max<int64_t>({c.d_model, hd, c.ffn_dim});
        chain(dev_alloc(&m->pf_h, (size_t)PF_ROWS * c.d_model));
        chain(dev_alloc(&m->pf_c, (size_t)PF_ROWS * nc));
        chain(dev_alloc(&m->pf_q, (size_t)PF_ROWS * hd));
        chain(dev_alloc(&m->pf_part, (size_t)PF_MAX_SPLITS * PF_ROWS * c.d_model));
        chain(dev_alloc(&m->pf_x, (size_t)X_TERMS * m->pf_term));
        m->pf_y_term = (int64_t)PF_ROWS * c.ffn_dim;
        chain(dev_alloc(&m->pf_y, (size_t)X_TERMS * m->pf_y_term));
    }
    if (st != SD_OK) {
        destroy_model(m);
        return st;
    }
    if (hipHostMalloc(reinterpret_cast<void **>(&m->mb_host), sizeof(Mailbox), hipHostMallocCoherent) !=
        hipSuccess) {
        m->mb_host = nullptr;
        destroy_model(m);
        return fail(SD_ERR_OOM, "pinned mailbox allocation failed");
    }
    std::memset(m->mb_host, 0, sizeof(Mailbox));
    if (hipHostGetDevicePointer(reinterpret_cast<void **>(&m->mb_dev), m->mb_host, 0) != hipSuccess) {
        destroy_model(m);
        return fail(SD_ERR_DEVICE, "mailbox device pointer failed");
    }
    for (hipEvent_t &e : m->ev)
        if (hipEventCreate(&e) != hipSuccess) {
            destroy_model(m);
            return fail(SD_ERR_DEVICE, "event creation failed");
        }
    // activations start at zero (rows beyond the current forward are read
    // as zeros by the 16-row kernels' padding lanes only through masks)
    if (hipMemsetAsync(ws.h, 0, sizeof(float) * (size_t)MAX_ROWS * c.d_model, m->stream) != hipSuccess ||
        hipMemsetAsync(ws.mbuf, 0, sizeof(float) * (size_t)MAX_ROWS * c.ffn_dim, m->stream) != hipSuccess ||
        hipMemsetAsync(ws.o, 0, sizeof(float) * (size_t)MAX_ROWS * c.n_heads * c.head_dim, m->stream) !=
            hipSuccess ||
        hipStreamSynchronize(m->stream) != hipSuccess) {
        destroy_model(m);
        return fail(SD_ERR_DEVICE, "workspace initialisation failed");
    }
    *out = m;
    return SD_OK;
}

// The kernel symbol of a plan as the profiler prints it.
std::string kernel_symbol(const sd_model *m, const Plan &p) {
    const char *tw = m->bf16 ? "unsigned short" : "float";
    const bool norm = p.kind == LK_QKV || p.kind == LK_GATE_UP || p.kind == LK_HEAD;
    if (p.path == PATH_MFMA) {
        // the packing count follows the row bound of each launch; name the
        // widest one the timed launches used
        const int hi = m->timed_rows_hi ? m->timed_rows_hi : MAX_ROWS;
        const int np = mfma_packs(hi);
        std::string nm = "void sdk::k_linear_mfma<" + std::to_string(p.epi) + ", " +
                         std::to_string(mfma_shape_tn(p.epi, np)) + ", " + std::to_string(mfma_shape_nw(p.epi, np)) +
                         ", " + std::to_string(np) + ">(sdk::LinearArgs)";
        if (m->timed_rows_lo && mfma_packs(m->timed_rows_lo) != mfma_packs(hi))
            nm += " (mixed packings)";
        return nm;
    }
    const int mr = p.path == PATH_GEMV
                       ? 1
                       : ((p.path == PATH_VALU2 || p.path == PATH_WAVE2) ? 2 : 16);
    const bool wave = p.path == PATH_WAVE2;
    const int nt = wave ? 64 : 256, u = wave ? (p.chunks ? p.chunks : wave2_default_chunks(p.rows)) : 1;
    return std::string("void sdk::k_linear_valu<") + tw + ", " + std::to_string(mr) + ", " + std::to_string(p.rows) +
           ", " + std::to_string(p.epi) + ", " + (norm ? "true" : "false") + ", " + std::to_string(nt) + ", " +
           std::to_string(u) + ">(sdk::LinearArgs)";
}

const Plan *find_plan(const sd_model *m, int kind, int regime) {
    if (kind < 0 || kind >= LK_COUNT)
        return nullptr;
    if (regime == 1)
        return &m->plan1[kind];
    if (regime == 2)
        return &m->plan2[kind];
    if (regime == 16)
        return &m->planm[kind];
    return nullptr;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI

#define SD_GUARD(body)                                                                                 \
    try {                                                                                              \
        body                                                                                           \
    } catch (const std::bad_alloc &) {                                                                 \
        return fail(SD_ERR_OOM, "host allocation failed");                                             \
    } catch (...) {                                                                                    \
        return fail(SD_ERR_DEVICE, "unexpected internal error");                                       \
    }

extern "C" {

sd_status sd_model_create(const sd_config *config, const sd_weights *weights, void *hip_stream, sd_model **out) {
    SD_GUARD(g_err.clear(); return create_model(config, weights, hip_stream, out);)
}

sd_status sd_model_destroy(sd_model *model) {
    SD_GUARD(if (!model) return fail(SD_ERR_INVALID_ARG, "model is null"); destroy_model(model); return SD_OK;)
}

size_t sd_kv_cache_bytes(const sd_config *config, int32_t capacity) {
    if (!config || capacity < 0 || check_config(config) != SD_OK)
        return 0;
    return kv_bytes(*config, capacity);
}

sd_status sd_kv_cache_create(sd_model *model, int32_t capacity, void *device_buf, sd_kv_cache **out) {
    SD_GUARD(if (!model || !out) return fail(SD_ERR_INVALID_ARG, "model or out is null");
             *out = nullptr; return create_user_cache(model, capacity, device_buf, out);)
}

sd_status sd_kv_cache_destroy(sd_kv_cache *cache) {
    SD_GUARD(if (!cache) return fail(SD_ERR_INVALID_ARG, "cache is null");
             destroy_user_cache(cache); return SD_OK;)
}

int32_t sd_kv_cache_length(const sd_kv_cache *cache) { return cache ? cache->len : -1; }

sd_status sd_kv_cache_truncate(sd_kv_cache *cache, int32_t len) {
    if (!cache)
        return fail(SD_ERR_INVALID_ARG, "cache is null");
    if (len < 0 || len > cache->len)
        return fail(SD_ERR_INVALID_ARG, "truncate length must be in [0, length]");
    cache->len = len;
    return SD_OK;
}

sd_status sd_kv_cache_set_length(sd_kv_cache *cache, int32_t len) {
    if (!cache)
        return fail(SD_ERR_INVALID_ARG, "cache is null");
    if (len < 0 || len > cache->cap)
        return fail(SD_ERR_CAPACITY, "length must be in [0, capacity]");
    cache->len = len;
    return SD_OK;
}

sd_status sd_forward(sd_model *model, const int32_t *tokens, int32_t n, const uint8_t *skip_mask,
                     sd_kv_cache *cache, float *logits) {
    SD_GUARD(return forward(model, tokens, n, skip_mask, cache, logits);)
}

sd_status sd_forward_static(sd_model *model, const int32_t *tokens, int32_t n, const uint8_t *skip_mask,
                            sd_kv_cache *cache, float *logits) {
    SD_GUARD(return forward_static(model, tokens, n, skip_mask, cache, logits);)
}

sd_status sd_model_quantize_draft(sd_model *model, const uint8_t *skip_mask) {
    SD_GUARD(return quantize_draft(model, skip_mask);)
}

sd_status sd_model_draft_fp8(const sd_model *model, int32_t layer, int32_t kind, const void **q,
                             const int32_t **exps) {
    SD_GUARD(if (!model || !q || !exps) return fail(SD_ERR_INVALID_ARG, "model, q or exps is null");
             if (layer < 0 || layer >= model->cfg.n_layers || kind < 0 || kind > 3)
                 return fail(SD_ERR_INVALID_ARG, "layer or kind out of range");
             *q = model->fp8_q[layer][kind]; *exps = model->fp8_e[layer][kind]; return SD_OK;)
}

sd_status sd_self_spec_generate(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                const uint8_t *skip_mask, int32_t K_max, float gamma, int32_t *out_tokens,
                                sd_stats *stats) {
    SD_GUARD(ExitRule rule{}; rule.gamma = gamma;
             return self_spec(model, prompt, prompt_len, max_new, skip_mask, K_max, rule, nullptr, out_tokens,
                              stats);)
}

sd_status sd_self_spec_generate_adaptive(sd_model *model, const int32_t *prompt, int32_t prompt_len,
                                         int32_t max_new, const uint8_t *skip_mask, int32_t K_max,
                                         const sd_adaptive *params, int32_t *out_tokens, sd_stats *stats) {
    SD_GUARD(if (!params) return fail(SD_ERR_INVALID_ARG, "params is null"); ExitRule rule{};
             rule.adaptive = 1; rule.gamma = (float)params->gamma0; rule.gamma0 = params->gamma0;
             rule.alpha = params->alpha; rule.epsilon = params->epsilon; rule.beta1 = params->beta1;
             rule.beta2 = params->beta2;
             return self_spec(model, prompt, prompt_len, max_new, skip_mask, K_max, rule, nullptr, out_tokens,
                              stats);)
}

sd_status sd_autoregressive_generate(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                     int32_t *out_tokens, sd_stats *stats) {
    SD_GUARD(return autoregressive(model, prompt, prompt_len, max_new, nullptr, out_tokens, stats);)
}

namespace {
SampleParams sample_params(const sd_sampling &s) {
    SampleParams p;
    p.temperature = s.temperature;
    p.top_p = s.top_p;
    p.seed = s.seed;
    return p;
}
ExitRule adaptive_rule(const sd_adaptive &a) {
    ExitRule r{};
    r.adaptive = 1;
    r.gamma = (float)a.gamma0;
    r.gamma0 = a.gamma0;
    r.alpha = a.alpha;
    r.epsilon = a.epsilon;
    r.beta1 = a.beta1;
    r.beta2 = a.beta2;
    return r;
}
}  // namespace

sd_status sd_self_spec_sample(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                              const uint8_t *skip_mask, int32_t K_max, float gamma, const sd_adaptive *adaptive,
                              const sd_sampling *sampling, int32_t *out_tokens, sd_stats *stats) {
    SD_GUARD(if (!sampling) return fail(SD_ERR_INVALID_ARG, "sampling is null"); ExitRule rule{};
             rule.gamma = gamma; if (adaptive) rule = adaptive_rule(*adaptive);
             const SampleParams sp = sample_params(*sampling);
             return self_spec(model, prompt, prompt_len, max_new, skip_mask, K_max, rule, &sp, out_tokens, stats);)
}

sd_status sd_autoregressive_sample(sd_model *model, const int32_t *prompt, int32_t prompt_len, int32_t max_new,
                                   const sd_sampling *sampling, int32_t *out_tokens, sd_stats *stats) {
    SD_GUARD(if (!sampling) return fail(SD_ERR_INVALID_ARG, "sampling is null");
             const SampleParams sp = sample_params(*sampling);
             return autoregressive(model, prompt, prompt_len, max_new, &sp, out_tokens, stats);)
}

sd_status sd_model_time_kernel(sd_model *model, int32_t layer, int32_t rows) {
    SD_GUARD(if (!model) return fail(SD_ERR_INVALID_ARG, "model is null");
             if (layer != -1 && !find_plan(model, layer, rows))
                 return fail(SD_ERR_INVALID_ARG, "layer must be -1 or 0..4 and rows 1, 2 or 16");
             model->timed_kind = layer; model->timed_regime = rows; model->tev_used = 0;
             model->timed_forwards = 0; model->timed_now = false;
             model->timed_rows_lo = 0; model->timed_rows_hi = 0;
             model->timed_launches = 0; model->timed_ms = 0.0; return SD_OK;)
}

sd_status sd_model_kernel_time(sd_model *model, int64_t *launches, double *total_ms, char *kernel_name,
                               int32_t name_cap, int64_t *n, int64_t *k) {
    SD_GUARD(if (!model) return fail(SD_ERR_INVALID_ARG, "model is null");
             const Plan *p = find_plan(model, model->timed_kind, model->timed_regime);
             if (launches) *launches = model->timed_launches;
             if (total_ms) *total_ms = model->timed_ms;
             if (n) *n = p ? p->N : 0;
             if (k) *k = p ? p->K : 0;
             if (kernel_name && name_cap > 0) {
                 const std::string nm = p ? kernel_symbol(model, *p) : std::string();
                 const size_t len = std::min<size_t>(nm.size(), (size_t)name_cap - 1);
                 std::memcpy(kernel_name, nm.data(), len);
                 kernel_name[len] = 0;
             } return SD_OK;)
}

const char *sd_last_error(void) { return g_err.c_str(); }

const char *sd_version(void) { return "sd-mi355x 0.1 (gfx950)"; }

}  // extern "C"

namespace sdk {

sd_status report(sd_status st, const std::string &msg) { return fail(st, msg); }

int32_t model_layers(const sd_model *m) { return m ? m->cfg.n_layers : 0; }

}  // namespace sdk
