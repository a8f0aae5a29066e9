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
__device__ inline uint64_t wfix(float w) { return (uint64_t)(w * WFIX); }  // exact scaling, truncation

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    return v;
}

// Block sum; red is LDS scratch of SWAVES words.  Integer: any order is exact.
__device__ uint64_t block_sum_u64(uint64_t v, uint64_t *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    v = wave_sum_u64(v);
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    uint64_t t = 0;
#pragma unroll
    for (int w = 0; w < SWAVES; ++w)
        t += red[w];
    __syncthreads();
    return t;
}

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
    for (int w = 0; w < SWAVES; ++w)
        t = fmaxf(t, red[w]);
    __syncthreads();
    return t;
}

// Exclusive prefix sum over the threads in thread order; *total receives the sum.
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
    for (int w = 0; w < SWAVES; ++w) {
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

__global__ __launch_bounds__(SW) void k_warp_rows(SampleArgs a, int mode) {
    __shared__ uint64_t red[SWAVES];
    __shared__ float redf[SWAVES];
    __shared__ uint64_t bins[SWAVES][16];
    __shared__ uint64_t bsum[16];
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
    for (int x = tid; x < V; x += SW)
        mx = fmaxf(mx, lg[x]);
    mx = block_max_f(mx, redf);
    uint64_t z = 0;
    for (int x = tid; x < V; x += SW)
        z += wfix(warp_w(lg[x], mx, T));
    z = block_sum_u64(z, red);

    uint32_t bstar = 0, n_tie = 0xffffffffu;
    uint64_t zs = z;
    if (a.sp.top_p < 1.0f) {
        // target mass: mass >= top_p * Z  <=>  mass >= ceil(top_p * Z) for integer masses
        uint64_t target = (uint64_t)ceil((double)a.sp.top_p * (double)z);
        target = target < 1 ? 1 : target;
        // Largest bit pattern b* with M(b*) >= target, M(b) = mass of w with bits >= b.
        // Invariant: M(lo) >= target > M(hi); m_hi = M(hi).
        uint32_t lo = 0, hi = 0x3f800001u;  // every weight is in (0, 1]
        uint64_t m_hi = 0;
        while (hi - lo > 1) {
            const uint32_t step = (hi - lo + 15) / 16;
            uint64_t acc[16];
#pragma unroll
            for (int i = 0; i < 16; ++i)
                acc[i] = 0;
            for (int x = tid; x < V; x += SW) {
                const float w = warp_w(lg[x], mx, T);
                const uint32_t b = __float_as_uint(w);
                if (b >= lo && b < hi) {
                    const uint32_t idx = (b - lo) / step;
                    const uint64_t W = wfix(w);
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        acc[i] += idx == (uint32_t)i ? W : 0;
                }
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const uint64_t v = wave_sum_u64(acc[i]);
                if (lane == 0)
                    bins[wave][i] = v;
            }
            __syncthreads();
            if (tid < 16) {
                uint64_t t = 0;
                for (int w = 0; w < SWAVES; ++w)
                    t += bins[w][tid];
                bsum[tid] = t;
            }
            __syncthreads();
            // largest sub-interval start t_i = lo + i step (below hi) with M(t_i) >= target
            uint64_t above = m_hi;  // M(t_{i+1}) while scanning down
            int best = 0;
            uint64_t m_next = m_hi;
            for (int i = 15; i >= 0; --i) {
                if (lo + (uint64_t)i * step >= hi)
                    continue;
                const uint64_t mi = above + bsum[i];
                if (mi >= target) {
                    best = i;
                    m_next = above;
                    break;
                }
                above = mi;
            }
            const uint64_t nh = (uint64_t)lo + (uint64_t)(best + 1) * step;
            hi = nh < hi ? (uint32_t)nh : hi;
            lo = lo + (uint32_t)best * step;
            m_hi = m_next;
            __syncthreads();  // bsum is rewritten by the next pass
        }
        bstar = lo;
        // the tokens at w*: all of them, or the lowest ids until the target
        uint64_t c_tie = 0;
        for (int x = tid; x < V; x += SW)
            c_tie += __float_as_uint(warp_w(lg[x], mx, T)) == bstar ? 1 : 0;
        c_tie = block_sum_u64(c_tie, red);
        const uint64_t wstar = wfix(__uint_as_float(bstar));
        uint64_t need = target - m_hi;  // > 0 by the invariant
        uint64_t nt = wstar == 0 ? c_tie : (need + wstar - 1) / wstar;
        nt = nt < c_tie ? nt : c_tie;
        n_tie = (uint32_t)nt;
        zs = m_hi + nt * wstar;
    }

    // a verification row: the weight of the draft it judges, if that draft is in the nucleus
    uint64_t wd = 0;
    if (mode == HEAD_VERIFY && r + 1 < M) {
        const int d = a.ctl->tokens[r + 1];
        const float w = warp_w(lg[d], mx, T);
        const uint32_t b = __float_as_uint(w);
        bool kept = b > bstar || n_tie == 0xffffffffu;
        if (!kept && b == bstar) {
            uint64_t rank = 0;  // ties with lower ids
            for (int x = tid; x < d; x += SW)
                rank += __float_as_uint(warp_w(lg[x], mx, T)) == bstar ? 1 : 0;
            rank = block_sum_u64(rank, red);
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

// The nucleus weight of token x of a row given its rank among the row's
// tokens at w* (only consulted for those).
struct RowView {
    const float *lg;
    float mx, T;
    uint32_t bstar, n_tie;
    __device__ uint64_t weight(int x, uint64_t &tie_rank, float *wout) const {
        const float w = warp_w(lg[x], mx, T);
        *wout = w;
        const uint32_t b = __float_as_uint(w);
        if (n_tie == 0xffffffffu || b > bstar)
            return wfix(w);
        if (b == bstar)
            return tie_rank++ < n_tie ? wfix(w) : 0;
        return 0;
    }
    __device__ bool is_tie(int x) const {
        return n_tie != 0xffffffffu && __float_as_uint(warp_w(lg[x], mx, T)) == bstar;
    }
};

__device__ RowView row_view(const float *lg, const RowStat &s, float T) {
    return RowView{lg, s.mx, T, s.bstar, s.n_tie};
}

// Inverse-CDF draw with uniform u24 / 2^24 over the weights of p (residual
// == false) or over fixed(max(0, p_x - q_x)) with p and q normalised by
// their nucleus masses (residual == true).  Returns the token, or -1 when
// every weight is zero; *wsel receives the chosen token's weight.
__device__ int block_draw(const RowView &p, uint64_t zs_p, const RowView &q, uint64_t zs_q, bool residual,
                          uint32_t u24, int V, uint64_t *wsel, uint64_t *red, int *sel, uint64_t *selw) {
    const int tid = threadIdx.x;
    const int seg = (V + SW - 1) / SW;
    const int x0 = min(V, tid * seg), x1 = min(V, x0 + seg);
    // ranks of this segment's first tie tokens in each row
    uint64_t tp = 0, tq = 0, tot;
    for (int x = x0; x < x1; ++x) {
        tp += p.is_tie(x) ? 1 : 0;
        if (residual)
            tq += q.is_tie(x) ? 1 : 0;
    }
    uint64_t rp0 = block_excl_scan_u64(tp, red, &tot);
    uint64_t rq0 = residual ? block_excl_scan_u64(tq, red, &tot) : 0;
    const float izp = WFIX / (float)zs_p, izq = residual ? WFIX / (float)zs_q : 0.0f;
    auto wt = [&](int x, uint64_t &rp, uint64_t &rq) -> uint64_t {
        float wp, wq;
        const uint64_t Wp = p.weight(x, rp, &wp);
        if (!residual)
            return Wp;
        const uint64_t Wq = q.weight(x, rq, &wq);
        const float px = Wp ? wp * izp : 0.0f, qx = Wq ? wq * izq : 0.0f;
        return wfix(fmaxf(px - qx, 0.0f));
    };
    uint64_t s = 0;
    {
        uint64_t rp = rp0, rq = rq0;
        for (int x = x0; x < x1; ++x)
            s += wt(x, rp, rq);
    }
    const uint64_t pre = block_excl_scan_u64(s, red, &tot);
    if (tid == 0)
        *sel = -1;
    __syncthreads();
    if (tot > 0) {
        // floor(u24 * total / 2^24): the draw is the first x whose cumulative mass exceeds it
        const uint64_t hi = __umul64hi((uint64_t)u24, tot), lo = (uint64_t)u24 * tot;
        const uint64_t thr = (hi << 40) | (lo >> 24);
        if (pre <= thr && thr < pre + s) {
            uint64_t c = pre, rp = rp0, rq = rq0;
            for (int x = x0; x < x1; ++x) {
                const uint64_t w = wt(x, rp, rq);
                c += w;
                if (c > thr) {
                    *sel = x;
                    *selw = w;
                    break;
                }
            }
        }
    }
    __syncthreads();
    const int x = *sel;
    *wsel = *selw;
    __syncthreads();
    return x;
}

// ---------------------------------------------------------------------------
// The decision of one step.

__global__ __launch_bounds__(SW) void k_sample_decide(SampleArgs a, int mode) {
    __shared__ uint64_t red[SWAVES];
    __shared__ int sel;
    __shared__ uint64_t selw;
    __shared__ int n_acc;
    const int tid = threadIdx.x, V = a.vocab;
    DevState *st = a.head.st;
    DevCtl *ctl = const_cast<DevCtl *>(a.ctl);
    const float T = a.sp.temperature;
    const uint64_t seed = a.sp.seed;
    const int e = st->emitted;
    uint64_t w;
    if (mode == HEAD_AR) {
        // token e of autoregressive sampling: counter (e, final draw, stage e)
        const RowStat s0 = a.vstat[0];
        const RowView p = row_view(a.vlog, s0, T);
        const int tok = block_draw(p, s0.zs, p, 0, false, uniform24(seed, e, U_FINAL, e), V, &w, red, &sel, &selw);
        if (tid == 0)
            ar_commit(a.head, ctl, tok);
    } else if (mode == HEAD_DRAFT) {
        const int j = st->k;
        const RowStat sj = a.dstat[j];
        const RowView q = row_view(a.dlog + (int64_t)j * V, sj, T);
        const int d = block_draw(q, sj.zs, q, 0, false, uniform24(seed, e + j, U_DRAFT, st->n_stages), V, &w, red,
                                 &sel, &selw);
        if (tid == 0) {
            st->dqw[j] = w;
            // the top token has weight exactly 2^40, so max q = 2^40 / mass
            draft_commit(a.head, ctl, d, (float)((double)WFIX / (double)sj.zs));
        }
    } else {
        const int k = st->k;
        const int64_t stage = st->n_stages;
        if (tid == 0) {
            int n = 0;
            for (; n < k; ++n) {
                const double r = (double)uniform24(seed, e + n, U_ACCEPT, stage) * 0x1p-24;
                const double pd = (double)a.vstat[n].wd / (double)a.vstat[n].zs;
                const double qd = (double)st->dqw[n] / (double)a.dstat[n].zs;
                const double ratio = pd / qd;
                if (!(r < (ratio < 1.0 ? ratio : 1.0)))
                    break;
            }
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
            tok = block_draw(p, sp.zs, q, sq.zs, true, u, V, &w, red, &sel, &selw);
            if (tok < 0)  // an empty residual (rounding): draw from p
                tok = block_draw(p, sp.zs, p, 0, false, u, V, &w, red, &sel, &selw);
        } else {
            tok = block_draw(p, sp.zs, p, 0, false, u, V, &w, red, &sel, &selw);
        }
        if (tid == 0)
            stage_commit(a.head, ctl, n, tok);
    }
}

hipError_t launch_sample_step(const SampleArgs &a, int max_rows, hipStream_t s) {
    const int mode = a.head.mode;
    if (mode != HEAD_AR && mode != HEAD_DRAFT && mode != HEAD_VERIFY)
        return hipErrorInvalidValue;
    if (max_rows < 1 || max_rows > MAX_ROWS || a.vocab < 1)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_warp_rows, dim3(mode == HEAD_VERIFY ? max_rows : 1), dim3(SW), 0, s, a, mode);
    hipLaunchKernelGGL(k_sample_decide, dim3(1), dim3(SW), 0, s, a, mode);
    return hipGetLastError();
}

}  // namespace sdk
