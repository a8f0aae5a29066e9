// Sampling variant of self-speculative decoding (the appendix's algorithm
// with random sampling): drafts are drawn from the warped draft distribution
// q, draft d is accepted when r < min(1, p(d) / q(d)) with p the warped
// full-model distribution, the first rejected position is redrawn from
// max(0, p - q) normalised, and a fully accepted stage ends with a draw from
// p.  The warping (temperature, top-p nucleus) and the fixed-point masses are
// described with RowStat in sd_internal.h.
//
// Two kernels follow the head linear, which has written the logits:
//   k_warp_rows     one work-group per row: max logit, total mass, the
//                   nucleus cut by a 16-ary search over the bit patterns of
//                   the float32 weights (positive floats order like their
//                   bits), and for a verification row the weight of the
//                   draft it judges;
//   k_sample_decide one work-group: the step's draws and acceptance tests in
//                   order, then the shared state update.
// Draws are inverse-CDF in id order over exact integer masses: a block-wide
// exclusive scan of per-thread segment masses finds the segment holding
// floor(u * total), and its thread walks the segment.
#include "sd_internal.h"
#include "decode_step.h"

namespace sdk {

constexpr int SW = 1024;         // threads of the sampling work-groups
constexpr int SWAVES = SW / 64;
// RowStat::n_tie when every token at w* is in the nucleus (no rank needed)
constexpr uint32_t ALL_TIES = 0xffffffffu;
// draws walk the vocabulary in chunks of DRAW_CHUNK ids, 8 adjacent ids per thread
constexpr int DRAW_CHUNK = 8 * SW;
constexpr int MAX_DRAW_CHUNKS = MAX_SAMPLE_VOCAB / DRAW_CHUNK;

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC'11), from its definition: ten rounds of
// (x0, x1, x2, x3) -> (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1,
// lo(M0 x0)), the key advanced by the Weyl constants between rounds.
// Returns the top 24 bits of the first output word: the uniform is u / 2^24.
__device__ inline uint32_t uniform24(uint64_t seed, int64_t index, int32_t purpose, int64_t stage) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    uint64_t x0 = (uint64_t)index, x1 = (uint64_t)(uint32_t)purpose, x2 = (uint64_t)stage, x3 = 0;
    uint64_t k0 = seed, k1 = 0;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t hi0 = __umul64hi(M0, x0), lo0 = M0 * x0;
        const uint64_t hi1 = __umul64hi(M1, x2), lo1 = M1 * x2;
        const uint64_t y0 = hi1 ^ x1 ^ k0, y2 = hi0 ^ x3 ^ k1;
        x0 = y0;
        x1 = lo1;
        x2 = y2;
        x3 = lo0;
    }
    return (uint32_t)(x0 >> 40);
}

__device__ inline float warp_w(float l, float mx, float T) { return expf((l - mx) / T); }
// fixed-point weight: exact scaling by 2^31, truncation; at most 2^31
__device__ inline uint32_t wfix(float w) { return (uint32_t)(w * WFIX); }

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    return v;
}

// Sums of 16 per-lane values over the 64 lanes of a wave by a transposing
// butterfly.  At the step over lane bit b (b = 5, 4, 3, 2) each lane keeps
// the half of its values selected by that bit and adds its partner's copy
// of them (8 + 4 + 2 + 1 shuffles); two plain steps over bits 1 and 0 then
// add the four lanes that hold the same value.  Lane l returns the wave's
// sum of value (l >> 2) & 15: 17 shuffles instead of 16 x 6.  Integer sums
// are exact in any order.
__device__ inline uint64_t wave_sum16_u64(const uint64_t (&acc)[16], int lane) {
    uint64_t a8[8], a4[4], a2[2];
    {
        const bool h = lane & 32;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            a8[j] = (h ? acc[8 + j] : acc[j]) + __shfl_xor(h ? acc[j] : acc[8 + j], 32, 64);
    }
    {
        const bool h = lane & 16;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            a4[j] = (h ? a8[4 + j] : a8[j]) + __shfl_xor(h ? a8[j] : a8[4 + j], 16, 64);
    }
    {
        const bool h = lane & 8;
#pragma unroll
        for (int j = 0; j < 2; ++j)
            a2[j] = (h ? a4[2 + j] : a4[j]) + __shfl_xor(h ? a4[j] : a4[2 + j], 8, 64);
    }
    const bool h = lane & 4;
    uint64_t a1 = (h ? a2[1] : a2[0]) + __shfl_xor(h ? a2[0] : a2[1], 4, 64);
    a1 += __shfl_xor(a1, 2, 64);
    a1 += __shfl_xor(a1, 1, 64);
    return a1;
}

// Block sum over NT threads; red is LDS scratch of NT / 64 words.  Integer:
// any order is exact.
template <int NT = SW>
__device__ uint64_t block_sum_u64(uint64_t v, uint64_t *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    v = wave_sum_u64(v);
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    uint64_t t = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w)
        t += red[w];
    __syncthreads();
    return t;
}

template <int NT = SW>
__device__ float block_max_f(float v, float *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v = fmaxf(v, __shfl_xor(v, o, 64));
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    float t = -INFINITY;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w)
        t = fmaxf(t, red[w]);
    __syncthreads();
    return t;
}

// Exclusive prefix sum over the NT threads in thread order; *total receives the sum.
template <int NT = SW>
__device__ uint64_t block_excl_scan_u64(uint64_t v, uint64_t *red, uint64_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t y = __shfl_up(x, o, 64);
        if (lane >= o)
            x += y;
    }
    if (lane == 63)
        red[wave] = x;
    __syncthreads();
    uint64_t base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        const uint64_t r = red[w];
        base += w < wave ? r : 0;
        tot += r;
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

// ---------------------------------------------------------------------------
// Nucleus statistics of one row per work-group.
//
// Element i of thread t is token t + i SW.  With EPT > 0 every thread keeps
// the weight bit patterns of its EPT tokens in registers (vocab <= EPT SW),
// computed once, and rebuilds the fixed-point weight from them; with
// EPT == 0 each pass recomputes both from the logits (any vocab).


template <int NT>
__device__ uint32_t block_min_u32(uint32_t v, uint64_t *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v = min(v, (uint32_t)__shfl_xor((int)v, o, 64));
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    uint32_t t = 0xffffffffu;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w)
        t = min(t, (uint32_t)red[w]);
    __syncthreads();
    return t;
}

// NT threads per row: 512 keeps up to 256 registers per lane, room for the
// cached patterns (EPT of them) and the 16 accumulators.
// Once at most CAND tokens lie in the search interval, their patterns move
// to LDS and the remaining passes read only those.
constexpr int CAND = 2048;

template <int NT, int EPT>
__global__ __launch_bounds__(NT) void k_warp_rows(SampleArgs a, int mode) {
    constexpr int NWV = NT / 64;
    __shared__ uint64_t red[NWV];
    __shared__ float redf[NWV];
    __shared__ uint64_t bins[NWV][16];
    __shared__ uint64_t bsum[16];
    __shared__ uint32_t cand[EPT > 0 ? CAND : 1];
    const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int M = a.ctl->m, V = a.vocab;
    if (r >= M)
        return;  // uniform over the work-group
    const bool draft = mode == HEAD_DRAFT;
    const int slot = draft ? a.head.st->k : r;
    const float *lg = (draft ? a.dlog : a.vlog) + (int64_t)slot * V;
    RowStat *out = (draft ? a.dstat : a.vstat) + slot;
    const float T = a.sp.temperature;

    float mx = -INFINITY;
    float lv[EPT > 0 ? EPT : 1];
    if constexpr (EPT > 0) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int x = tid + i * NT;
            lv[i] = x < V ? lg[x] : -INFINITY;
            mx = fmaxf(mx, lv[i]);
        }
    } else {
        for (int x = tid; x < V; x += NT)
            mx = fmaxf(mx, lg[x]);
    }
    mx = block_max_f<NT>(mx, redf);
    uint32_t cb[EPT > 0 ? EPT : 1];  // weight bit patterns (padding: weight 0)
    uint64_t z = 0;
    uint32_t bmin = 0xffffffffu;
    if constexpr (EPT > 0) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const float w = tid + i * NT < V ? warp_w(lv[i], mx, T) : 0.0f;
            cb[i] = __float_as_uint(w);
            z += wfix(w);
            bmin = tid + i * NT < V ? min(bmin, cb[i]) : bmin;
        }
    } else {
        for (int x = tid; x < V; x += NT) {
            const float w = warp_w(lg[x], mx, T);
            z += wfix(w);
            bmin = min(bmin, __float_as_uint(w));
        }
    }
    z = block_sum_u64<NT>(z, red);

    uint32_t bstar = 0, n_tie = ALL_TIES;  // top_p = 1: every token (pattern >= 0)
    uint64_t zs = z;
    if (a.sp.top_p < 1.0f) {
        // target mass: mass >= top_p * Z  <=>  mass >= ceil(top_p * Z) for integer masses
        uint64_t target = (uint64_t)ceil((double)a.sp.top_p * (double)z);
        target = target < 1 ? 1 : target;
        // Largest bit pattern b* with M(b*) >= target, M(b) = mass of w with bits >= b.
        // Invariant: M(lo) >= target > M(hi); m_hi = M(hi).  Every weight's
        // pattern is in [min pattern, pattern of 1.0].
        uint32_t lo = block_min_u32<NT>(bmin, red), hi = 0x3f800001u;
        uint64_t m_hi = 0;
        bool compacted = false;  // the interval's patterns are cand[0, ncand)
        int ncand = 0;
        while (hi - lo > 1) {
            // lo, hi and step are the same in every thread: keep them scalar
            lo = __builtin_amdgcn_readfirstlane(lo);
            hi = __builtin_amdgcn_readfirstlane(hi);
            const uint32_t step = __builtin_amdgcn_readfirstlane((hi - lo + 15) / 16);
            // acc_i = mass of the tokens with lo + i step <= bits < hi, so
            // M(lo + i step) = m_hi + acc_i (thresholds at or past hi stay 0)
            uint64_t acc[16];
#pragma unroll
            for (int i = 0; i < 16; ++i)
                acc[i] = 0;
            auto add = [&](uint32_t b) {
                if (b >= lo && b < hi) {
                    const uint32_t d = b - lo, W = wfix(__uint_as_float(b));
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        acc[i] += d >= (uint32_t)i * step ? W : 0u;
                }
            };
            if constexpr (EPT > 0) {
                if (compacted) {
                    for (int k = tid; k < ncand; k += NT)
                        add(cand[k]);
                } else {
#pragma unroll
                    for (int i = 0; i < EPT; ++i)
                        if (tid + i * NT < V)
                            add(cb[i]);
                }
            } else {
                for (int x = tid; x < V; x += NT)
                    add(__float_as_uint(warp_w(lg[x], mx, T)));
            }
            {
                const uint64_t v = wave_sum16_u64(acc, lane);
                if ((lane & 3) == 0)
                    bins[wave][lane >> 2] = v;
            }
            __syncthreads();
            if (tid < 16) {
                uint64_t t = 0;
                for (int w = 0; w < NWV; ++w)
                    t += bins[w][tid];
                bsum[tid] = t;
            }
            __syncthreads();
            // largest threshold t_i below hi with M(t_i) >= target (t_0 = lo qualifies)
            int best = 0;
            for (int i = 15; i > 0; --i) {
                if (lo + (uint64_t)i * step < hi && m_hi + bsum[i] >= target) {
                    best = i;
                    break;
                }
            }
            const uint64_t m_next = best < 15 && lo + (uint64_t)(best + 1) * step < hi ? m_hi + bsum[best + 1] : m_hi;
            const uint64_t nh = (uint64_t)lo + (uint64_t)(best + 1) * step;
            hi = nh < hi ? (uint32_t)nh : hi;
            lo = lo + (uint32_t)best * step;
            m_hi = m_next;
            __syncthreads();  // bsum is rewritten by the next pass
            if constexpr (EPT > 0) {
                if (!compacted && hi - lo > 1) {
                    uint64_t n = 0;
#pragma unroll
                    for (int i = 0; i < EPT; ++i)
                        n += (tid + i * NT < V && cb[i] >= lo && cb[i] < hi) ? 1 : 0;
                    uint64_t tot;
                    uint64_t pos = block_excl_scan_u64<NT>(n, red, &tot);
                    if (tot <= CAND) {  // uniform
#pragma unroll
                        for (int i = 0; i < EPT; ++i)
                            if (tid + i * NT < V && cb[i] >= lo && cb[i] < hi)
                                cand[pos++] = cb[i];
                        compacted = true;
                        ncand = (int)tot;
                        __syncthreads();
                    }
                }
            }
        }
        bstar = lo;
        // the tokens at w*: all of them, or the lowest ids until the target
        uint64_t c_tie = 0;
        if constexpr (EPT > 0) {
#pragma unroll
            for (int i = 0; i < EPT; ++i)
                c_tie += (tid + i * NT < V && cb[i] == bstar) ? 1 : 0;
        } else {
            for (int x = tid; x < V; x += NT)
                c_tie += __float_as_uint(warp_w(lg[x], mx, T)) == bstar ? 1 : 0;
        }
        c_tie = block_sum_u64<NT>(c_tie, red);
        const uint64_t wstar = wfix(__uint_as_float(bstar));
        uint64_t need = target - m_hi;  // > 0 by the invariant
        uint64_t nt = wstar == 0 ? c_tie : (need + wstar - 1) / wstar;
        nt = nt < c_tie ? nt : c_tie;
        n_tie = nt == c_tie ? ALL_TIES : (uint32_t)nt;
        zs = m_hi + nt * wstar;
    }

    // a verification row: the weight of the draft it judges, if that draft is in the nucleus
    uint64_t wd = 0;
    if (mode == HEAD_VERIFY && r + 1 < M) {
        const int d = a.ctl->tokens[r + 1];
        const float w = warp_w(lg[d], mx, T);
        const uint32_t b = __float_as_uint(w);
        bool kept = b > bstar || (b == bstar && n_tie == ALL_TIES);
        if (!kept && b == bstar) {
            uint64_t rank = 0;  // ties with lower ids
            for (int x = tid; x < d; x += NT)
                rank += __float_as_uint(warp_w(lg[x], mx, T)) == bstar ? 1 : 0;
            rank = block_sum_u64<NT>(rank, red);
            kept = rank < n_tie;
        }
        wd = kept ? wfix(w) : 0;
    }
    if (tid == 0) {
        RowStat st;
        st.mx = mx;
        st.bstar = bstar;
        st.n_tie = n_tie;
        st.pad = 0;
        st.zs = zs;
        st.wd = wd;
        *out = st;
    }
}

// ---------------------------------------------------------------------------
// Draws.

// A row's nucleus: token x is in it when its weight pattern exceeds b*, or
// equals b* and, unless every such token is, its rank among them by id is
// below n_tie.
struct RowView {
    const float *lg;
    float mx, T;
    uint32_t bstar, n_tie;
    __device__ bool partial() const { return n_tie != ALL_TIES; }
    // weight of x (0 outside the nucleus); tie_rank counts the ties seen
    __device__ uint32_t weight(int x, uint32_t &tie_rank, float *wout) const {
        const float w = warp_w(lg[x], mx, T);
        *wout = w;
        const uint32_t b = __float_as_uint(w);
        if (b > bstar)
            return wfix(w);
        if (b == bstar)
            return (!partial() || tie_rank++ < n_tie) ? wfix(w) : 0u;
        return 0u;
    }
    __device__ bool is_tie(int x) const { return __float_as_uint(warp_w(lg[x], mx, T)) == bstar; }
};

__device__ RowView row_view(const float *lg, const RowStat &s, float T) {
    return RowView{lg, s.mx, T, s.bstar, s.n_tie};
}

struct DrawScratch {
    uint64_t red[SWAVES];
    uint64_t chunk_tot[MAX_DRAW_CHUNKS];
    uint32_t tie_p[MAX_DRAW_CHUNKS], tie_q[MAX_DRAW_CHUNKS];  // ties before each chunk
    int sel;
    uint32_t selw;
};

// Inverse-CDF draw with uniform u24 / 2^24 over the nucleus weights of p
// (residual == false) or over fixed(max(0, p_x - q_x)), p and q normalised by
// their nucleus masses (residual == true), in id order.  Chunk j holds ids
// [j DRAW_CHUNK, (j + 1) DRAW_CHUNK); thread t its ids j DRAW_CHUNK + 8 t ..
// + 7.  The chunk totals locate the draw; one exclusive scan inside that
// chunk locates the thread, which walks its 8 ids.  Ranks among ties are
// followed only when a row cuts its ties.  Returns the token, or -1 when
// every weight is zero; *wsel receives the chosen token's weight.
__device__ int block_draw(const RowView &p, uint64_t zs_p, const RowView &q, uint64_t zs_q, bool residual,
                          uint32_t u24, int V, uint32_t *wsel, DrawScratch &sc) {
    const int tid = threadIdx.x;
    const int nchunks = (V + DRAW_CHUNK - 1) / DRAW_CHUNK;
    const bool ranks = p.partial() || (residual && q.partial());
    const float izp = WFIX / (float)zs_p, izq = residual ? WFIX / (float)zs_q : 0.0f;
    auto wt = [&](int x, uint32_t &rp, uint32_t &rq) -> uint32_t {
        float wp, wq;
        const uint32_t Wp = p.weight(x, rp, &wp);
        if (!residual)
            return Wp;
        const uint32_t Wq = q.weight(x, rq, &wq);
        const float px = Wp ? wp * izp : 0.0f, qx = Wq ? wq * izq : 0.0f;
        return wfix(fmaxf(px - qx, 0.0f));
    };
    // pass 1: chunk totals (and, with ranks, the ties before each chunk and thread)
    uint32_t tp_run = 0, tq_run = 0;
    uint64_t total = 0, tot;
    for (int j = 0; j < nchunks; ++j) {
        const int x0 = j * DRAW_CHUNK + 8 * tid, x1 = min(V, x0 + 8);
        uint32_t rp = 0, rq = 0;
        if (ranks) {
            uint32_t cp = 0, cq = 0;
            for (int x = x0; x < x1; ++x) {
                cp += p.partial() && p.is_tie(x) ? 1 : 0;
                cq += residual && q.partial() && q.is_tie(x) ? 1 : 0;
            }
            const uint64_t pp = block_excl_scan_u64(cp, sc.red, &tot);
            if (tid == 0)
                sc.tie_p[j] = tp_run;
            rp = tp_run + (uint32_t)pp;
            tp_run += (uint32_t)tot;
            const uint64_t pq = block_excl_scan_u64(cq, sc.red, &tot);
            if (tid == 0)
                sc.tie_q[j] = tq_run;
            rq = tq_run + (uint32_t)pq;
            tq_run += (uint32_t)tot;
        }
        uint64_t s = 0;
        for (int x = x0; x < x1; ++x)
            s += wt(x, rp, rq);
        s = block_sum_u64(s, sc.red);
        if (tid == 0)
            sc.chunk_tot[j] = s;
        total += s;
    }
    if (tid == 0)
        sc.sel = -1;
    __syncthreads();
    if (total > 0) {
        // floor(u24 * total / 2^24): the draw is the first x whose cumulative mass exceeds it
        const uint64_t hi = __umul64hi((uint64_t)u24, total), lo = (uint64_t)u24 * total;
        const uint64_t thr = (hi << 40) | (lo >> 24);
        int js = 0;
        uint64_t before = 0;
        while (js + 1 < nchunks && before + sc.chunk_tot[js] <= thr)
            before += sc.chunk_tot[js++];
        // pass 2, chunk js only: this thread's 8 ids
        const int x0 = js * DRAW_CHUNK + 8 * tid, x1 = min(V, x0 + 8);
        uint32_t rp0 = 0, rq0 = 0;
        if (ranks) {
            uint32_t cp = 0, cq = 0;
            for (int x = x0; x < x1; ++x) {
                cp += p.partial() && p.is_tie(x) ? 1 : 0;
                cq += residual && q.partial() && q.is_tie(x) ? 1 : 0;
            }
            rp0 = sc.tie_p[js] + (uint32_t)block_excl_scan_u64(cp, sc.red, &tot);
            rq0 = sc.tie_q[js] + (uint32_t)block_excl_scan_u64(cq, sc.red, &tot);
        }
        uint64_t s = 0;
        {
            uint32_t rp = rp0, rq = rq0;
            for (int x = x0; x < x1; ++x)
                s += wt(x, rp, rq);
        }
        const uint64_t pre = before + block_excl_scan_u64(s, sc.red, &tot);
        if (pre <= thr && thr < pre + s) {
            uint64_t c = pre;
            uint32_t rp = rp0, rq = rq0;
            for (int x = x0; x < x1; ++x) {
                const uint32_t w = wt(x, rp, rq);
                c += w;
                if (c > thr) {
                    sc.sel = x;
                    sc.selw = w;
                    break;
                }
            }
        }
    }
    __syncthreads();
    const int x = sc.sel;
    *wsel = sc.selw;
    __syncthreads();
    return x;
}

// ---------------------------------------------------------------------------
// The decision of one step.

__global__ __launch_bounds__(SW) void k_sample_decide(SampleArgs a, int mode) {
    __shared__ DrawScratch sc;
    __shared__ int n_acc;
    __shared__ bool acc_ok[MAX_ROWS];
    const int tid = threadIdx.x, V = a.vocab;
    DevState *st = a.head.st;
    DevCtl *ctl = const_cast<DevCtl *>(a.ctl);
    if (ctl->m == 0)
        return;  // a cancelled step takes no decision
    const float T = a.sp.temperature;
    const uint64_t seed = a.sp.seed;
    const int e = st->emitted;
    uint32_t w;
    if (mode == HEAD_AR) {
        // token e of autoregressive sampling: counter (e, final draw, stage e)
        const RowStat s0 = a.vstat[0];
        const RowView p = row_view(a.vlog, s0, T);
        const int tok = block_draw(p, s0.zs, p, 0, false, uniform24(seed, e, U_FINAL, e), V, &w, sc);
        if (tid == 0)
            ar_commit(a.head, ctl, tok);
    } else if (mode == HEAD_DRAFT) {
        const int j = st->k;
        const RowStat sj = a.dstat[j];
        const RowView q = row_view(a.dlog + (int64_t)j * V, sj, T);
        const int d = block_draw(q, sj.zs, q, 0, false, uniform24(seed, e + j, U_DRAFT, st->n_stages), V, &w, sc);
        if (tid == 0) {
            st->dqw[j] = w;
            // the top token has weight exactly WFIX, so max q = WFIX / mass
            draft_commit(a.head, ctl, d, (float)((double)WFIX / (double)sj.zs));
        }
    } else {
        const int k = st->k;
        const int64_t stage = st->n_stages;
        // draft i is accepted when r_i < min(1, p_i(d) / q_i(d)); thread i
        // evaluates test i, thread 0 finds the first failure
        if (tid < k) {
            const double r = (double)uniform24(seed, e + tid, U_ACCEPT, stage) * 0x1p-24;
            const double pd = (double)a.vstat[tid].wd / (double)a.vstat[tid].zs;
            const double qd = (double)st->dqw[tid] / (double)a.dstat[tid].zs;
            const double ratio = pd / qd;
            acc_ok[tid] = r < (ratio < 1.0 ? ratio : 1.0);
        }
        __syncthreads();
        if (tid == 0) {
            int n = 0;
            while (n < k && acc_ok[n])
                ++n;
            n_acc = n;
        }
        __syncthreads();
        const int n = n_acc;
        const uint32_t u = uniform24(seed, e + n, U_FINAL, stage);
        const RowStat sp = a.vstat[n];
        const RowView p = row_view(a.vlog + (int64_t)n * V, sp, T);
        int tok;
        if (n < k) {
            const RowStat sq = a.dstat[n];
            const RowView q = row_view(a.dlog + (int64_t)n * V, sq, T);
            tok = block_draw(p, sp.zs, q, sq.zs, true, u, V, &w, sc);
            if (tok < 0)  // an empty residual (rounding): draw from p
                tok = block_draw(p, sp.zs, p, 0, false, u, V, &w, sc);
        } else {
            tok = block_draw(p, sp.zs, p, 0, false, u, V, &w, sc);
        }
        if (tid == 0)
            stage_commit(a.head, ctl, n, tok);
    }
}

hipError_t launch_sample_step(const SampleArgs &a, int max_rows, hipStream_t s) {
    const int mode = a.head.mode;
    if (mode != HEAD_AR && mode != HEAD_DRAFT && mode != HEAD_VERIFY)
        return hipErrorInvalidValue;
    if (max_rows < 1 || max_rows > MAX_ROWS || a.vocab < 1 || a.vocab > MAX_DRAW_CHUNKS * DRAW_CHUNK)
        return hipErrorInvalidValue;
    const dim3 grid(mode == HEAD_VERIFY ? max_rows : 1);
    if (a.vocab <= 64 * 512)
        hipLaunchKernelGGL((k_warp_rows<512, 64>), grid, dim3(512), 0, s, a, mode);
    else
        hipLaunchKernelGGL((k_warp_rows<SW, 0>), grid, dim3(SW), 0, s, a, mode);
    hipLaunchKernelGGL(k_sample_decide, dim3(1), dim3(SW), 0, s, a, mode);
    return hipGetLastError();
}

}  // namespace sdk
