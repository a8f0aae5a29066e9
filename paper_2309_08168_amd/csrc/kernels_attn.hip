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
// g are staged in LDS as float32; the queries of the g-th head group, all
// rows, attend to them 16 query vectors at a time.  Each (query, split)
// leaves a partial softmax state (max, sum of exp, unnormalised output).
template <typename TK>
__global__ __launch_bounds__(256) void k_attn_split(AttnArgs a) {
    constexpr int CH = ATTN_CHUNK;
    constexpr int DMAX = MAX_HEAD_DIM;
    __shared__ float Ks[CH][DMAX + 4];
    __shared__ float Vs[CH][DMAX];
    __shared__ float Qs[16][DMAX];
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
        load8_kv(Kg + (int64_t)key * dh + e, &Ks[key][e]);
        load8_kv(Vg + (int64_t)key * dh + e, &Vs[key][e]);
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
        for (int p = tid; p < nq * CH; p += 256) {
            const int qi = p / CH, c = p - qi * CH;
            const int r = (qg + qi) / G;
            float sres = -INFINITY;
            if (c < nk && c0 + c <= pos + r) {
                float acc = 0.0f;
                for (int e = 0; e < dh; e += 4) {
                    const float4 kv = *reinterpret_cast<const float4 *>(&Ks[c][e]);
                    const float4 qv = *reinterpret_cast<const float4 *>(&Qs[qi][e]);
                    acc = fmaf(qv.x, kv.x, acc);
                    acc = fmaf(qv.y, kv.y, acc);
                    acc = fmaf(qv.z, kv.z, acc);
                    acc = fmaf(qv.w, kv.w, acc);
                }
                sres = acc;
            }
            Ss[qi][c] = sres;
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
                acc = fmaf(Ss[qi][c], Vs[c][e], acc);
            const int qidx = qg + qi, r = qidx / G, head = g * G + (qidx - r * G);
            const int64_t slot = ((int64_t)split * H + head) * MAX_ROWS + r;
            a.part_o[slot * dh + e] = acc;
            if (e == 0)
                a.part_ml[slot] = MLs[qi];
        }
    }
}

// Ordered combine of the split partials of one (head, row): deterministic.
__global__ __launch_bounds__(128) void k_attn_combine(AttnArgs a) {
    const int head = blockIdx.x, r = blockIdx.y;
    const int pos = a.ctl->pos, M = a.ctl->m;
    if (r >= M)
        return;
    const int ns = (pos + M + ATTN_CHUNK - 1) / ATTN_CHUNK;
    const int dh = a.head_dim, H = a.n_heads;
    float mx = -INFINITY;
    for (int s = 0; s < ns; ++s)
        mx = fmaxf(mx, a.part_ml[((int64_t)s * H + head) * MAX_ROWS + r].x);
    for (int e = threadIdx.x; e < dh; e += blockDim.x) {
        float L = 0.0f, O = 0.0f;
        for (int s = 0; s < ns; ++s) {
            const int64_t slot = ((int64_t)s * H + head) * MAX_ROWS + r;
            const float2 ml = a.part_ml[slot];
            if (ml.x == -INFINITY)
                continue;
            const float w = expf(ml.x - mx);
            L = fmaf(w, ml.y, L);
            O = fmaf(w, a.part_o[slot * dh + e], O);
        }
        a.out[(int64_t)r * a.ld_out + (int64_t)head * dh + e] = O / L;
    }
}

hipError_t launch_attention(const AttnArgs &a, bool bf16, hipStream_t s) {
    if (a.head_dim > MAX_HEAD_DIM || (a.head_dim & 7))
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
