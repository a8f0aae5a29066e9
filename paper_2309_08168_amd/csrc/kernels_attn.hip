// Split-KV causal attention of 1..16 query rows over the KV cache, with
// grouped-query heads, plus the small kernels of a forward (embedding
// gather, control block, decode-state setup).
//
// Verification runs the full model over the last committed token and the
// drafts in one forward (Algorithm 2); row r of that block sits at position
// pos + r and sees keys 0..pos + r, including the K/V the same forward just
// appended.  A draft step is the one-row case.
#include "sd_internal.h"

namespace sdk {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void load8_kv(const uint16_t *p, float *dst) {
    const u32x4_t v = *reinterpret_cast<const u32x4_t *>(p);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        dst[2 * j] = __uint_as_float(v[j] << 16);
        dst[2 * j + 1] = __uint_as_float(v[j] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8_kv(const float *p, float *dst) {
    const f32x4_t a = reinterpret_cast<const f32x4_t *>(p)[0];
    const f32x4_t b = reinterpret_cast<const f32x4_t *>(p)[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        dst[j] = a[j];
        dst[4 + j] = b[j];
    }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_add(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    return v;
}

// Work-group (split, kv head g): keys [split * CH, split * CH + CH) of head
// g are staged in LDS in the cache's storage type; the queries of the g-th
// head group, all rows, attend to them 16 query vectors at a time.  Each
// (query, split) leaves a partial softmax state (max, sum of exp,
// unnormalised output).  The last work-group of head group g to finish
// (counted by a self-resetting counter) combines the splits of every query
// in split order, so the result is deterministic.
template <typename TK>
struct KvLds;
template <>
struct KvLds<uint16_t> {
    static constexpr int PAD = 8;
    __device__ static void load8(const uint16_t *src, uint16_t *dst) {
        *reinterpret_cast<u32x4_t *>(dst) = *reinterpret_cast<const u32x4_t *>(src);
    }
    __device__ static void read8(const uint16_t *p, float *v) {
        const u32x4_t w = *reinterpret_cast<const u32x4_t *>(p);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = __uint_as_float(w[j] << 16);
            v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
        }
    }
    __device__ static float read1(const uint16_t *p) { return __uint_as_float(((uint32_t)*p) << 16); }
};
template <>
struct KvLds<float> {
    static constexpr int PAD = 4;
    __device__ static void load8(const float *src, float *dst) {
        reinterpret_cast<f32x4_t *>(dst)[0] = reinterpret_cast<const f32x4_t *>(src)[0];
        reinterpret_cast<f32x4_t *>(dst)[1] = reinterpret_cast<const f32x4_t *>(src)[1];
    }
    __device__ static void read8(const float *p, float *v) {
        const f32x4_t a = reinterpret_cast<const f32x4_t *>(p)[0];
        const f32x4_t b = reinterpret_cast<const f32x4_t *>(p)[1];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[j] = a[j];
            v[4 + j] = b[j];
        }
    }
    __device__ static float read1(const float *p) { return *p; }
};

template <typename TK>
__global__ __launch_bounds__(256) void k_attn_split(AttnArgs a) {
    constexpr int CH = ATTN_CHUNK;
    constexpr int DMAX = MAX_HEAD_DIM;
    constexpr int KS = DMAX + KvLds<TK>::PAD;
    __shared__ __attribute__((aligned(16))) TK Ks[CH * KS];
    __shared__ __attribute__((aligned(16))) TK Vs[CH * DMAX];
    __shared__ __attribute__((aligned(16))) float Qs[16][DMAX];
    __shared__ float Ss[16][CH];
    __shared__ float2 MLs[16];
    const int split = blockIdx.x, g = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int pos = a.ctl->pos, M = a.ctl->m;
    const int ctx = pos + M;
    const int c0 = split * CH;
    if (c0 >= ctx)
        return;
    const int nk = min(CH, ctx - c0);
    const int dh = a.head_dim, H = a.n_heads;
    const int G = H / a.n_kv_heads;
    const int Q = G * M;

    const TK *Kg = reinterpret_cast<const TK *>(a.kcache) + (int64_t)g * a.kv_head_stride + (int64_t)c0 * dh;
    const TK *Vg = reinterpret_cast<const TK *>(a.vcache) + (int64_t)g * a.kv_head_stride + (int64_t)c0 * dh;
    const int d8 = dh >> 3;
    for (int i = tid; i < nk * d8; i += 256) {
        const int key = i / d8, e = (i - key * d8) * 8;
        KvLds<TK>::load8(Kg + (int64_t)key * dh + e, &Ks[key * KS + e]);
        KvLds<TK>::load8(Vg + (int64_t)key * dh + e, &Vs[key * DMAX + e]);
    }
    const float scale = 1.0f / sqrtf((float)dh);

    for (int qg = 0; qg < Q; qg += 16) {
        const int nq = min(16, Q - qg);
        __syncthreads();
        for (int i = tid; i < nq * dh; i += 256) {
            const int qi = i / dh, e = i - qi * dh;
            const int qidx = qg + qi, r = qidx / G, head = g * G + (qidx - r * G);
            Qs[qi][e] = a.q[(int64_t)r * a.ld_q + (int64_t)head * dh + e] * scale;
        }
        __syncthreads();
        // scores: thread (key c, query lane ql) takes queries ql, ql + 4, ...
        {
            const int c = tid & (CH - 1), ql = tid >> 6;
            float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if (c < nk && ql < nq) {
                for (int e = 0; e < dh; e += 8) {
                    float kv[8];
                    KvLds<TK>::read8(&Ks[c * KS + e], kv);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int qi = ql + 4 * u;
                        if (qi < nq) {
                            const float4 q0 = *reinterpret_cast<const float4 *>(&Qs[qi][e]);
                            const float4 q1 = *reinterpret_cast<const float4 *>(&Qs[qi][e + 4]);
                            float s = acc[u];
                            s = fmaf(q0.x, kv[0], s);
                            s = fmaf(q0.y, kv[1], s);
                            s = fmaf(q0.z, kv[2], s);
                            s = fmaf(q0.w, kv[3], s);
                            s = fmaf(q1.x, kv[4], s);
                            s = fmaf(q1.y, kv[5], s);
                            s = fmaf(q1.z, kv[6], s);
                            s = fmaf(q1.w, kv[7], s);
                            acc[u] = s;
                        }
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int qi = ql + 4 * u;
                if (qi < nq) {
                    const int r = (qg + qi) / G;
                    Ss[qi][c] = (c < nk && c0 + c <= pos + r) ? acc[u] : -INFINITY;
                }
            }
        }
        __syncthreads();
        for (int qi = wave; qi < nq; qi += 4) {
            const float v = Ss[qi][lane];
            const float mx = wave_max(v);
            const float e = (mx == -INFINITY) ? 0.0f : expf(v - mx);
            const float l = wave_add(e);
            Ss[qi][lane] = e;
            if (lane == 0)
                MLs[qi] = make_float2(mx, l);
        }
        __syncthreads();
        for (int i = tid; i < nq * dh; i += 256) {
            const int qi = i / dh, e = i - qi * dh;
            float acc = 0.0f;
            for (int c = 0; c < nk; ++c)
                acc = fmaf(Ss[qi][c], KvLds<TK>::read1(&Vs[c * DMAX + e]), acc);
            const int qidx = qg + qi, r = qidx / G, head = g * G + (qidx - r * G);
            const int64_t slot = ((int64_t)split * H + head) * MAX_ROWS + r;
            a.part_o[slot * dh + e] = acc;
            if (e == 0)
                a.part_ml[slot] = MLs[qi];
        }
    }

}

// Ordered combine of the split partials of one (head, row): deterministic.
// The running maxima and sums of all splits are loaded in parallel first.
__global__ __launch_bounds__(128) void k_attn_combine(AttnArgs a) {
    __shared__ float w_s[MAX_SPLITS];
    __shared__ float2 ml_s[MAX_SPLITS];
    __shared__ float red[2];
    const int head = blockIdx.x, r = blockIdx.y;
    const int pos = a.ctl->pos, M = a.ctl->m;
    if (r >= M)
        return;
    const int ns = (pos + M + ATTN_CHUNK - 1) / ATTN_CHUNK;
    const int dh = a.head_dim, H = a.n_heads, tid = threadIdx.x;
    float mx = -INFINITY;
    for (int sp = tid; sp < ns; sp += 128) {
        const float2 v = a.part_ml[((int64_t)sp * H + head) * MAX_ROWS + r];
        ml_s[sp] = v;
        mx = fmaxf(mx, v.x);
    }
    mx = wave_max(mx);
    if ((tid & 63) == 0)
        red[tid >> 6] = mx;
    __syncthreads();
    mx = fmaxf(red[0], red[1]);
    for (int sp = tid; sp < ns; sp += 128) {
        const float2 v = ml_s[sp];
        w_s[sp] = v.x == -INFINITY ? 0.0f : expf(v.x - mx);
    }
    __syncthreads();
    float L = 0.0f;
    for (int sp = 0; sp < ns; ++sp)
        L = fmaf(w_s[sp], ml_s[sp].y, L);
    for (int e = tid; e < dh; e += 128) {
        float O = 0.0f;
        int sp = 0;
        for (; sp + 8 <= ns; sp += 8) {
            float ov[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                ov[u] = a.part_o[(((int64_t)(sp + u) * H + head) * MAX_ROWS + r) * dh + e];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                O = fmaf(w_s[sp + u], ov[u], O);
        }
        for (; sp < ns; ++sp)
            O = fmaf(w_s[sp], a.part_o[(((int64_t)sp * H + head) * MAX_ROWS + r) * dh + e], O);
        const float y = O / L;
        const int64_t oi = (int64_t)r * a.ld_out + (int64_t)head * dh + e;
        if (a.out_hi) {
            const uint32_t b = __float_as_uint(y);
            a.out_hi[oi] = (uint16_t)(b >> 16);
            a.out_lo[oi] = (uint16_t)(__float_as_uint(y - __uint_as_float(b & 0xffff0000u)) >> 16);
        } else {
            a.out[oi] = y;
        }
    }
}

hipError_t launch_attention(const AttnArgs &a, bool bf16, hipStream_t s) {
    if (a.head_dim > MAX_HEAD_DIM || (a.head_dim & 7) || a.splits > MAX_SPLITS)
        return hipErrorInvalidValue;
    dim3 grid(a.splits, a.n_kv_heads), block(256);
    if (bf16)
        hipLaunchKernelGGL(k_attn_split<uint16_t>, grid, block, 0, s, a);
    else
        hipLaunchKernelGGL(k_attn_split<float>, grid, block, 0, s, a);
    hipLaunchKernelGGL(k_attn_combine, dim3(a.n_heads, MAX_ROWS), dim3(128), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// small kernels

template <typename TW>
__global__ __launch_bounds__(256) void k_embed(const TW *E, int d, const DevCtl *ctl, float *h, int64_t ldh) {
    const int r = blockIdx.x;
    if (r >= ctl->m)
        return;
    const int64_t tok = ctl->tokens[r];
    for (int i = threadIdx.x; i < d; i += 256) {
        float v;
        if constexpr (sizeof(TW) == 2)
            v = __uint_as_float(((uint32_t)E[tok * d + i]) << 16);
        else
            v = E[tok * d + i];
        h[(int64_t)r * ldh + i] = v;
    }
}

hipError_t launch_embed(const void *emb, bool bf16, int d, const DevCtl *ctl, float *h, int64_t ldh,
                        hipStream_t s) {
    if (bf16)
        hipLaunchKernelGGL(k_embed<uint16_t>, dim3(MAX_ROWS), dim3(256), 0, s,
                           reinterpret_cast<const uint16_t *>(emb), d, ctl, h, ldh);
    else
        hipLaunchKernelGGL(k_embed<float>, dim3(MAX_ROWS), dim3(256), 0, s, reinterpret_cast<const float *>(emb),
                           d, ctl, h, ldh);
    return hipGetLastError();
}

__global__ void k_set_ctl(DevCtl *ctl, int32_t pos, int32_t m, const int32_t *tokens) {
    const int i = threadIdx.x;
    if (i == 0) {
        ctl->pos = pos;
        ctl->m = m;
    }
    if (i < m)
        ctl->tokens[i] = tokens[i];
}

hipError_t launch_set_ctl(DevCtl *ctl, int32_t pos, int32_t m, const int32_t *dev_tokens, hipStream_t s) {
    hipLaunchKernelGGL(k_set_ctl, dim3(1), dim3(64), 0, s, ctl, pos, m, dev_tokens);
    return hipGetLastError();
}

// State at the start of decoding: the cache holds the prompt minus its last
// token; the first stage drafts from that last token.
__global__ void k_init_decode(DevState *st, DevCtl *ctl, Mailbox *mb, int32_t lc, const int32_t *last,
                              int32_t max_new, int32_t k_max, float gamma) {
    if (threadIdx.x != 0)
        return;
    const int tok = *last;
    st->lc = lc;
    st->last = tok;
    st->emitted = 0;
    st->max_new = max_new;
    st->k = 0;
    st->k_max = k_max;
    const int kcap = min(k_max, max_new - 1);
    st->kcap = kcap;
    st->phase = kcap > 0 ? PHASE_DRAFT : PHASE_VERIFY;
    st->gen_done = max_new <= 0;
    st->seq = 0;
    st->gamma = gamma;
    st->n_stages = st->n_drafted = st->n_accepted = st->n_draft_steps = 0;
    ctl->pos = lc;
    ctl->m = 1;
    ctl->tokens[0] = tok;
    if (mb) {
        __hip_atomic_store(&mb->phase, st->phase, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(&mb->gen_done, st->gen_done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(&mb->emitted, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(&mb->seq, 0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

hipError_t launch_init_decode(DevState *st, DevCtl *ctl, Mailbox *mb, int32_t lc, const int32_t *dev_last,
                              int32_t max_new, int32_t k_max, float gamma, hipStream_t s) {
    hipLaunchKernelGGL(k_init_decode, dim3(1), dim3(64), 0, s, st, ctl, mb, lc, dev_last, max_new, k_max, gamma);
    return hipGetLastError();
}

__global__ void k_fill_zero(uint32_t *p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

hipError_t launch_fill_zero(void *p, size_t bytes, hipStream_t s) {
    const size_t n = bytes / 4;
    if (n == 0)
        return hipSuccess;
    const unsigned blocks = (unsigned)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
    hipLaunchKernelGGL(k_fill_zero, dim3(blocks), dim3(256), 0, s, reinterpret_cast<uint32_t *>(p), n);
    return hipGetLastError();
}

}  // namespace sdk
