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

__device__ __forceinline__ void unpack8_bf16(u32x4_t v, float (&w)[8]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        w[2 * j] = __uint_as_float(v[j] << 16);
        w[2 * j + 1] = __uint_as_float(v[j] & 0xffff0000u);
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

// One work-group per (chunk of ATTN_CHUNK keys, kv head g), split-KV
// flash decoding.  Each of the AW waves takes 16 consecutive keys; its lanes
// form 4 groups of 16, group j holds keys j, j + 4, j + 8, j + 12 and lane
// e16 of a group holds head_dim / 16 consecutive elements of q, K and V, so
// each K or V row is one coalesced load by 16 lanes.  A wave keeps its K and
// V in registers (32 VGPRs for bf16 at head_dim 128), which leaves room for
// several waves per SIMD: a decode step has only c * head_dim * 4 bytes of
// KV per kv head to read, and small work-groups spread it over every CU.
// For up to QB query vectors at a time, every group scores its 4 keys, the
// four groups' softmax states merge by shuffles, the AW waves' states merge
// in LDS in wave order, and the chunk leaves one partial state per (query,
// split) for the ordered combine.
//
// Loads are unconditional: the caller passes the address of a valid cache
// row (clamped into the context) and a flag that zeroes the values after
// the load.  A load under a branch would make the compiler wait for every
// outstanding load where the branches join, serialising the round trips.
template <typename TK, int ED>
struct KvFrag {
    float v[ED];
    __device__ __forceinline__ void load(const TK *p, bool ok) {
        if constexpr (sizeof(TK) == 2) {
#pragma unroll
            for (int e = 0; e < ED; ++e) {
                const float x = __uint_as_float(((uint32_t)reinterpret_cast<const uint16_t *>(p)[e]) << 16);
                v[e] = ok ? x : 0.0f;
            }
        } else {
#pragma unroll
            for (int e = 0; e < ED; ++e) {
                const float x = reinterpret_cast<const float *>(p)[e];
                v[e] = ok ? x : 0.0f;
            }
        }
    }
    __device__ __forceinline__ float at(int e) const { return v[e]; }
};
// bf16 rows of 8 elements stay packed (16 bytes) until used
template <>
struct KvFrag<uint16_t, 8> {
    u32x4_t w;
    __device__ __forceinline__ void load(const uint16_t *p, bool ok) {
        const u32x4_t x = *reinterpret_cast<const u32x4_t *>(p);
        w = ok ? x : u32x4_t{0u, 0u, 0u, 0u};
    }
    __device__ __forceinline__ float at(int e) const {
        const uint32_t x = w[e >> 1];
        return __uint_as_float((e & 1) ? (x & 0xffff0000u) : (x << 16));
    }
};

constexpr int AW = 8;                  // waves per chunk
constexpr int AKW = ATTN_CHUNK / AW;   // keys per wave
static_assert(AKW == 16, "a wave holds 4 keys per lane group");

template <typename TK, int ED, int QB>
__global__ __launch_bounds__(AW * 64) void k_attn_split(AttnArgs a) {
    constexpr int KPG = AKW / 4;  // keys per lane group
    __shared__ float red_o[AW][QB][MAX_HEAD_DIM];
    __shared__ float2 red_ml[AW][QB];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int split = blockIdx.x, g = blockIdx.y;
    const int pos = a.ctl->pos, M = a.ctl->m;
    const int ctx = pos + M;
    const int c0 = split * ATTN_CHUNK;
    if (M == 0 || c0 >= ctx)
        return;  // uniform over the work-group (M = 0: a cancelled step)
    const int dh = a.head_dim, H = a.n_heads;
    const int G = H / a.n_kv_heads;
    const int Q = G * M;
    const int ks = lane >> 4, e16 = lane & 15;
    const int cw = c0 + wave * AKW;  // first key of this wave
    const TK *Kg = reinterpret_cast<const TK *>(a.kcache) + (int64_t)g * a.kv_head_stride + (int64_t)cw * dh + e16 * ED;
    const TK *Vg = reinterpret_cast<const TK *>(a.vcache) + (int64_t)g * a.kv_head_stride + (int64_t)cw * dh + e16 * ED;
    const float scale = 1.0f / sqrtf((float)dh);

    KvFrag<TK, ED> kf[KPG], vf[KPG];
#pragma unroll
    for (int j = 0; j < KPG; ++j) {
        const int c = ks + 4 * j;
        const bool ok = cw + c < ctx;
        const int cc = ok ? c : ctx - 1 - cw;  // a row inside the context
        kf[j].load(Kg + (int64_t)cc * dh, ok);
        vf[j].load(Vg + (int64_t)cc * dh, ok);
    }
    // Query vector qidx (one past the last reads the first).  Passes of one
    // or two vectors load them with the K/V rows; wider passes load each
    // vector where it is used, which keeps fewer registers live.
    auto load_q = [&](int qidx, float(&qv)[ED]) {
        qidx = qidx < Q ? qidx : 0;
        const int r = qidx / G, head = g * G + (qidx - r * G);
        const float *qs = a.q + (int64_t)r * a.ld_q + (int64_t)head * dh + e16 * ED;
#pragma unroll
        for (int e = 0; e < ED; ++e)
            qv[e] = qs[e] * scale;
    };
    constexpr bool PRELOAD = QB <= 2;
    float qb[PRELOAD ? QB : 1][ED];
    if constexpr (PRELOAD) {
#pragma unroll
        for (int qi = 0; qi < QB; ++qi)
            load_q(qi, qb[qi]);
    }
    // every load above is issued before the first result is waited for
    __builtin_amdgcn_sched_barrier(0);

    for (int qg = 0; qg < Q; qg += QB) {
        const int nq = min(QB, Q - qg);
        if (PRELOAD && qg) {
#pragma unroll
            for (int qi = 0; qi < (PRELOAD ? QB : 1); ++qi)
                load_q(qg + qi, qb[qi]);
        }
#pragma unroll
        for (int qi = 0; qi < QB; ++qi) {
            if (qi >= nq)
                break;
            const int qidx = qg + qi, r = qidx / G;
            float qv[ED];
            if constexpr (PRELOAD) {
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    qv[e] = qb[qi][e];
            } else {
                load_q(qidx, qv);
            }
            const int lim = pos + r - cw;  // last key row r sees, relative to the wave
            float s[KPG];
            float mx = -INFINITY;
#pragma unroll
            for (int j = 0; j < KPG; ++j) {
                float t = 0.0f;
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    t = fmaf(qv[e], kf[j].at(e), t);
                t += __shfl_xor(t, 1, 64);
                t += __shfl_xor(t, 2, 64);
                t += __shfl_xor(t, 4, 64);
                t += __shfl_xor(t, 8, 64);
                const int c = ks + 4 * j;
                s[j] = (cw + c < ctx && c <= lim) ? t : -INFINITY;
                mx = fmaxf(mx, s[j]);
            }
            float l = 0.0f, o[ED];
#pragma unroll
            for (int e = 0; e < ED; ++e)
                o[e] = 0.0f;
            if (mx != -INFINITY) {
#pragma unroll
                for (int j = 0; j < KPG; ++j) {
                    const float p = expf(s[j] - mx);
                    l += p;
#pragma unroll
                    for (int e = 0; e < ED; ++e)
                        o[e] = fmaf(p, vf[j].at(e), o[e]);
                }
            }
            // merge the four key groups
#pragma unroll
            for (int x = 16; x <= 32; x <<= 1) {
                const float m2 = __shfl_xor(mx, x, 64), l2 = __shfl_xor(l, x, 64);
                float o2[ED];
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    o2[e] = __shfl_xor(o[e], x, 64);
                const float mn = fmaxf(mx, m2);
                if (mn != -INFINITY) {
                    const float wa = expf(mx - mn), wb = expf(m2 - mn);
                    l = l * wa + l2 * wb;
#pragma unroll
                    for (int e = 0; e < ED; ++e)
                        o[e] = o[e] * wa + o2[e] * wb;
                    mx = mn;
                }
            }
            if (ks == 0) {
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    red_o[wave][qi][e16 * ED + e] = o[e];
                if (e16 == 0)
                    red_ml[wave][qi] = make_float2(mx, l);
            }
        }
        __syncthreads();
        // merge the waves in wave order; one (query, element) per thread
        for (int t = threadIdx.x; t < nq * dh; t += AW * 64) {
            const int qi = t / dh, e = t - qi * dh;
            float m = -INFINITY;
#pragma unroll
            for (int w = 0; w < AW; ++w)
                m = fmaxf(m, red_ml[w][qi].x);
            float L = 0.0f, O = 0.0f;
            if (m != -INFINITY) {
#pragma unroll
                for (int w = 0; w < AW; ++w) {
                    const float2 ml = red_ml[w][qi];
                    if (ml.x != -INFINITY) {
                        const float wt = expf(ml.x - m);
                        L = fmaf(wt, ml.y, L);
                        O = fmaf(wt, red_o[w][qi][e], O);
                    }
                }
            }
            const int qidx = qg + qi, r = qidx / G, head = g * G + (qidx - r * G);
            const int64_t slot = ((int64_t)split * H + head) * MAX_ROWS + r;
            a.part_o[slot * dh + e] = O;
            if (e == 0)
                a.part_ml[slot] = make_float2(m, L);
        }
        __syncthreads();
    }
}

// The same split-KV attention on matrix cores, for bfloat16 caches and any
// number of query vectors: one work-group per (128-key chunk, kv head, tile
// of 16 query vectors), each of its 4 waves taking 32 keys.
//
// Scores S^T[key][q] = sum_e K[key][e] q[e] are 16x16x32 bf16 MFMAs with K
// rows as the A operand, read straight from the cache, and q (float32, times
// 1/sqrt(head_dim)) as the B operand, split into three bf16 terms that add
// up to it exactly, so every product is exact and only the float32
// accumulation rounds.  Row i of score tile t holds key 16 t + 4 (i % 4) +
// i / 4 of the wave: after the MFMA, lane group G (lanes 16 G..16 G + 15)
// then holds, for its query column, the keys 16 t + 4 v + G (v = 0..3), which
// are exactly the eight reduction slots 8 G + 4 t + v the output MFMA takes
// from that lane, so softmax weights never move between lanes.
//
// Outputs O^T[e][q] = sum_key V[key][e] P[q][key] are 16x16x32 MFMAs with
// P (split into three bf16 terms likewise) as the B operand and V^T as the A
// operand: the wave's 32 V rows are stored to a wave-private LDS tile with
// coalesced 16-byte loads and read back transposed (ds_read_b64_tr_b16, two
// reads per output tile), from rows padded by 32 bytes.  The softmax
// of a wave's 32 keys needs one cross-lane max and sum (lanes 16 apart); the
// four waves merge in LDS in wave order and the chunk leaves one partial per
// (query, split) for the ordered combine.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int MW = 4;                  // waves per work-group
constexpr int MKW = ATTN_CHUNK / MW;   // keys per wave
static_assert(MKW == 32, "a wave's keys are two 16-key score tiles");

__device__ __forceinline__ u32x4_t pack_bf16x8(const uint16_t (&h)[8]) {
    u32x4_t v;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        v[j] = (uint32_t)h[2 * j] | ((uint32_t)h[2 * j + 1] << 16);
    return v;
}

// Three bf16 terms of 8 float32 values, packed as MFMA operands.
__device__ __forceinline__ void split3x8(const float (&x)[8], u32x4_t (&t)[X_TERMS]) {
    uint16_t h[X_TERMS][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        uint16_t s[X_TERMS];
        split3(x[u], s);
#pragma unroll
        for (int i = 0; i < X_TERMS; ++i)
            h[i][u] = s[i];
    }
#pragma unroll
    for (int i = 0; i < X_TERMS; ++i)
        t[i] = pack_bf16x8(h[i]);
}

__device__ __forceinline__ f32x4_t mfma_bf16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

template <int DH>
__global__ __launch_bounds__(MW * 64) void k_attn_mfma(AttnArgs a) {
    constexpr int ES = DH / 32;            // 32-wide slices of head_dim (score MFMAs)
    constexpr int ET = DH / 16;            // 16-wide tiles of head_dim (output MFMAs)
    constexpr int VP = DH + 16;            // LDS pitch of a V row, bf16 elements
    constexpr int LPR = DH / 8;            // lanes per V row in 16-byte loads
    constexpr int RPI = 64 / LPR;          // V rows per load instruction
    constexpr int NVJ = MKW / RPI;         // V loads per lane
    constexpr int OP = 17;                 // LDS pitch of the merged output, floats per e
    constexpr int WB_V = MKW * VP * 2, WB_O = DH * OP * 4;
    constexpr int WS = (WB_V > WB_O ? WB_V : WB_O) / 4;  // words of one wave's LDS tile
    static_assert(WS % 2 == 0 && (VP * 2) % 8 == 0, "8-byte aligned rows for the transposed reads");
    __shared__ __attribute__((aligned(16))) uint32_t tile[MW][WS];
    __shared__ float2 red_ml[MW][16];

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int split = blockIdx.x, g = blockIdx.y, qt = blockIdx.z;
    const int pos = a.ctl->pos, M = a.ctl->m;
    const int ctx = pos + M;
    const int H = a.n_heads, G = H / a.n_kv_heads, Q = G * M;
    const int c0 = split * ATTN_CHUNK;
    if (M == 0 || c0 >= ctx || qt * 16 >= Q)
        return;  // uniform over the work-group (M = 0: a cancelled step)
    const int cw = c0 + wave * MKW;  // first key of this wave
    const int col = lane & 15, grp = lane >> 4;
    const uint16_t *Kg = reinterpret_cast<const uint16_t *>(a.kcache) + (int64_t)g * a.kv_head_stride;
    const uint16_t *Vg = reinterpret_cast<const uint16_t *>(a.vcache) + (int64_t)g * a.kv_head_stride;

    // query column col of this tile: row r of head g G + (qi mod G)
    const int qi = qt * 16 + col;
    const bool qok = qi < Q;
    const int r = qok ? qi / G : 0;
    const int head = g * G + (qi - r * G);
    // a column past the query vectors reads the first one and scores zero
    f32x4_t qraw[ES][2];
    {
        const float *qs = a.q + (qok ? (int64_t)r * a.ld_q + (int64_t)head * DH : (int64_t)g * G * DH) + 8 * grp;
#pragma unroll
        for (int s = 0; s < ES; ++s) {
            qraw[s][0] = reinterpret_cast<const f32x4_t *>(qs + 32 * s)[0];
            qraw[s][1] = reinterpret_cast<const f32x4_t *>(qs + 32 * s)[1];
        }
    }
    // K operands (A of the score MFMAs) and the wave's V rows.  Keys past the
    // context read the last row inside it: their scores are masked and their
    // weights are zero, and the row read is a finite one.
    u32x4_t kf[2][ES], vr[NVJ];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int key = min(cw + 16 * t + 4 * (col & 3) + (col >> 2), ctx - 1);
        const uint16_t *kp = Kg + (int64_t)key * DH + 8 * grp;
#pragma unroll
        for (int s = 0; s < ES; ++s)
            kf[t][s] = *reinterpret_cast<const u32x4_t *>(kp + 32 * s);
    }
#pragma unroll
    for (int j = 0; j < NVJ; ++j) {
        const int key = min(cw + j * RPI + lane / LPR, ctx - 1);
        vr[j] = *reinterpret_cast<const u32x4_t *>(Vg + (int64_t)key * DH + 8 * (lane % LPR));
    }
    // every load above is issued before the first result is waited for
    __builtin_amdgcn_sched_barrier(0);
    float qx[ES][8];
    {
        const float scale = 1.0f / sqrtf((float)DH);
#pragma unroll
        for (int s = 0; s < ES; ++s)
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                qx[s][u] = qok ? qraw[s][0][u] * scale : 0.0f;
                qx[s][4 + u] = qok ? qraw[s][1][u] * scale : 0.0f;
            }
    }

    // scores of the wave's 32 keys for query column col
    f32x4_t sacc[2];
    {
        u32x4_t qf[ES][X_TERMS];
#pragma unroll
        for (int s = 0; s < ES; ++s)
            split3x8(qx[s], qf[s]);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            sacc[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int s = 0; s < ES; ++s)
#pragma unroll
                for (int i = 0; i < X_TERMS; ++i)
                    sacc[t] = mfma_bf16(kf[t][s], qf[s][i], sacc[t]);
        }
    }
    // softmax over those keys; slot u = 4 t + v of this lane is key 16 t + 4 v + grp
    const int lim = pos + r;  // last key row r sees
    float sv[8], mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int key = cw + 16 * (u >> 2) + 4 * (u & 3) + grp;
        sv[u] = (qok && key < ctx && key <= lim) ? sacc[u >> 2][u & 3] : -INFINITY;
        mx = fmaxf(mx, sv[u]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float p[8], ls = 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        p[u] = mx == -INFINITY ? 0.0f : expf(sv[u] - mx);
        ls += p[u];
    }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    u32x4_t pf[X_TERMS];
    split3x8(p, pf);

    // V rows into the wave's LDS tile, then O^T = V^T P^T tile by tile
    uint16_t *vs = reinterpret_cast<uint16_t *>(tile[wave]);
#pragma unroll
    for (int j = 0; j < NVJ; ++j)
        *reinterpret_cast<u32x4_t *>(vs + (j * RPI + lane / LPR) * VP + 8 * (lane % LPR)) = vr[j];
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    f32x4_t oacc[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et) {
        // A operand V^T: lane (col, grp) needs column 16 et + col of keys
        // 16 (u >> 2) + 4 (u & 3) + grp, u = 0..7 (the score slots).
        // ds_read_b64_tr_b16 hands lane l of each 16-lane group element l % 4
        // of the 8 bytes that lanes l / 4 + 4 k (k = 0..3) point at, so lane
        // r points at key 16 I + 4 (r >> 2) + grp, columns 16 et + 4 (r & 3)
        // ..: two reads give the eight keys in order.
        uint32_t w[4];
#pragma unroll
        for (int I = 0; I < 2; ++I) {
            const uint16_t *src = vs + (16 * I + 4 * (col >> 2) + grp) * VP + 16 * et + 4 * (col & 3);
            const s16x4_t rv = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)src);
            w[2 * I] = (uint32_t)(uint16_t)rv[0] | ((uint32_t)(uint16_t)rv[1] << 16);
            w[2 * I + 1] = (uint32_t)(uint16_t)rv[2] | ((uint32_t)(uint16_t)rv[3] << 16);
        }
        const u32x4_t vf = {w[0], w[1], w[2], w[3]};
        oacc[et] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < X_TERMS; ++i)
            oacc[et] = mfma_bf16(vf, pf[i], oacc[et]);
    }
    // this wave's (max, sum, O^T) into its tile, which the V rows no longer need
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    float *ro = reinterpret_cast<float *>(tile[wave]);
#pragma unroll
    for (int et = 0; et < ET; ++et)
#pragma unroll
        for (int v = 0; v < 4; ++v)
            ro[(16 * et + 4 * grp + v) * OP + col] = oacc[et][v];
    if (grp == 0)
        red_ml[wave][col] = make_float2(mx, ls);
    __syncthreads();
    // merge the waves in wave order: the weight of each wave's state per
    // query column first (16 threads), then one (query, element) per thread.
    // A wave whose keys are all masked has weight 0 and an all-zero output.
    __shared__ float wts[MW][16];
    __shared__ float2 mls[16];
    if (threadIdx.x < 16) {
        const int qc = threadIdx.x;
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < MW; ++w)
            m = fmaxf(m, red_ml[w][qc].x);
        float L = 0.0f;
#pragma unroll
        for (int w = 0; w < MW; ++w) {
            const float2 ml = red_ml[w][qc];
            float wt = 0.0f;
            if (m != -INFINITY && ml.x != -INFINITY) {
                wt = expf(ml.x - m);
                L = fmaf(wt, ml.y, L);
            }
            wts[w][qc] = wt;
        }
        mls[qc] = make_float2(m, L);
    }
    __syncthreads();
    for (int t = threadIdx.x; t < 16 * DH; t += MW * 64) {
        const int qc = t / DH, e = t - qc * DH;
        const int qj = qt * 16 + qc;
        if (qj >= Q)
            break;  // t only grows
        float O = 0.0f;
#pragma unroll
        for (int w = 0; w < MW; ++w)
            O = fmaf(wts[w][qc], reinterpret_cast<const float *>(tile[w])[e * OP + qc], O);
        const int rj = qj / G, hj = g * G + (qj - rj * G);
        const int64_t slot = ((int64_t)split * H + hj) * MAX_ROWS + rj;
        a.part_o[slot * DH + e] = O;
        if (e == 0)
            a.part_ml[slot] = mls[qc];
    }
}

// Decode attention of one or two query vectors per kv head (the draft,
// autoregressive and one-draft verification steps of multi-head attention)
// over a bfloat16 cache with head_dim 128, on the VALU: one work-group of
// two waves per (64-key chunk, kv head), 32 keys per wave.
//
// Lane group j4 (lanes 16 j4 .. 16 j4 + 15) holds the key rows
// cw + 4 i + j4 (i = 0..7) of its wave and lane e16 of the group the
// elements 8 e16 .. 8 e16 + 7 of each row, so every K and V load
// instruction reads four whole rows (1 KB, coalesced).  A lane's partial
// dot products of its 8 rows are summed over the 16 lanes of the group by a
// butterfly over lane bits 3, 2, 1 that leaves row 4 b1 + 2 b2 + b3 in each
// lane (b = the lane's bits), then a quad exchange over bit 0: one score
// per lane, each key in two lanes.  The softmax of the wave's 32 keys is a
// whole-wave max and sum; the weights go through LDS to the lanes that hold
// the V rows, whose products are summed over the four groups by a butterfly
// over lane bits 5, 4 (two output elements per lane).  The two waves merge
// in LDS in wave order and the chunk leaves one partial state per (query,
// split) for the ordered combine.  Keys past the context read the last row
// inside it and are masked.
//
// The V rows are requested after the scores: with the K and V rows of a
// wave (16 loads per lane) requested at once, the short burst of a decode
// step streamed markedly slower (measured: a plain read of the same 26 MB
// with 16 loads in flight per thread took 8.7 us against 5.8 us with 4), and
// small work-groups spread it better (13B, 1280 keys, one row: 8.3 us with
// four waves of 32 keys and every load at once, 7.0 us like this).
constexpr int VW = 2;
static_assert(ATTN_CHUNK_VALU == VW * 32, "32 keys per wave");

template <int QV>
__global__ __launch_bounds__(VW * 64) void k_attn_valu(AttnArgs a) {
    constexpr int DH = 128;
    __shared__ float sp[VW][QV][32];
    __shared__ float so[VW][QV][DH];
    __shared__ float2 sml[VW][QV];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int j4 = lane >> 4, e16 = lane & 15;
    const int split = blockIdx.x, g = blockIdx.y;
    const int pos = a.ctl->pos, M = a.ctl->m;
    const int ctx = pos + M;
    const int H = a.n_heads, G = H / a.n_kv_heads, Q = G * M;
    const int c0 = split * ATTN_CHUNK_VALU;
    if (M == 0 || c0 >= ctx)
        return;  // uniform over the work-group (M = 0: a cancelled step)
    const int cw = c0 + wave * 32;
    const uint16_t *Kg = reinterpret_cast<const uint16_t *>(a.kcache) + (int64_t)g * a.kv_head_stride + 8 * e16;
    const uint16_t *Vg = reinterpret_cast<const uint16_t *>(a.vcache) + (int64_t)g * a.kv_head_stride + 8 * e16;

    // query vector qi: row qi / G, head g G + qi % G; a vector past Q reads
    // the first one and is masked
    f32x4_t qraw[QV][2];
#pragma unroll
    for (int qi = 0; qi < QV; ++qi) {
        const int qidx = qi < Q ? qi : 0, r = qidx / G;
        const float *qs = a.q + (int64_t)r * a.ld_q + (int64_t)(g * G + qidx - r * G) * DH + 8 * e16;
        qraw[qi][0] = reinterpret_cast<const f32x4_t *>(qs)[0];
        qraw[qi][1] = reinterpret_cast<const f32x4_t *>(qs)[1];
    }
    int keyrow[8];
    u32x4_t kr[8], vr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        keyrow[i] = min(cw + 4 * i + j4, ctx - 1);
        kr[i] = *reinterpret_cast<const u32x4_t *>(Kg + (int64_t)keyrow[i] * DH);
    }
    __builtin_amdgcn_sched_barrier(0);

    const float scale = 1.0f / sqrtf((float)DH);
    float s[QV][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float kx[8];
        unpack8_bf16(kr[i], kx);
#pragma unroll
        for (int qi = 0; qi < QV; ++qi) {
            float t = 0.0f;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                t = fmaf(qraw[qi][0][u] * scale, kx[u], t);
                t = fmaf(qraw[qi][1][u] * scale, kx[4 + u], t);
            }
            s[qi][i] = t;
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
        vr[i] = *reinterpret_cast<const u32x4_t *>(Vg + (int64_t)keyrow[i] * DH);
    const int b0 = lane & 1, b1 = (lane >> 1) & 1, b2 = (lane >> 2) & 1, b3 = (lane >> 3) & 1;
    const int row = 4 * b1 + 2 * b2 + b3;  // the row whose score this lane ends with
    const int key = cw + 4 * row + j4;
    float mx[QV], ls[QV];
#pragma unroll
    for (int qi = 0; qi < QV; ++qi) {
        float x4[4], x2[2];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            x4[u] = bfly8(s[qi][2 * u], s[qi][2 * u + 1], lane);
#pragma unroll
        for (int u = 0; u < 2; ++u)
            x2[u] = bfly4(x4[2 * u], x4[2 * u + 1], lane);
        float t = bfly2(x2[0], x2[1], lane);
        t += dpp_mov<DPP_QUAD_XOR1>(t);
        const int r = qi < Q ? qi / G : 0;
        const bool ok = qi < Q && key < ctx && key <= pos + r;
        const float sv = ok ? t : -INFINITY;
        mx[qi] = wave_max_all(sv);
        const float p = mx[qi] == -INFINITY ? 0.0f : expf(sv - mx[qi]);
        ls[qi] = wave_sum_all(b0 ? 0.0f : p);
        if (!b0)
            sp[wave][qi][8 * j4 + row] = p;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    // O = sum over the rows of p V, for the lane's 8 elements
    float o[QV][8];
#pragma unroll
    for (int qi = 0; qi < QV; ++qi)
#pragma unroll
        for (int u = 0; u < 8; ++u)
            o[qi][u] = 0.0f;
#pragma unroll
    for (int qi = 0; qi < QV; ++qi) {
        const f32x4_t pa = *reinterpret_cast<const f32x4_t *>(&sp[wave][qi][8 * j4]);
        const f32x4_t pb = *reinterpret_cast<const f32x4_t *>(&sp[wave][qi][8 * j4 + 4]);
        const float pw[8] = {pa[0], pa[1], pa[2], pa[3], pb[0], pb[1], pb[2], pb[3]};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float vx[8];
            unpack8_bf16(vr[i], vx);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                o[qi][u] = fmaf(pw[i], vx[u], o[qi][u]);
        }
    }
#pragma unroll
    for (int qi = 0; qi < QV; ++qi) {
        float y4[4], y2[2];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            y4[u] = bfly32(o[qi][2 * u], o[qi][2 * u + 1]);
#pragma unroll
        for (int u = 0; u < 2; ++u)
            y2[u] = bfly16(y4[2 * u], y4[2 * u + 1]);
        // element 8 e16 + 4 u + 2 b4 + b5 of the wave's output
        const int e0 = 8 * e16 + 2 * ((lane >> 4) & 1) + ((lane >> 5) & 1);
        so[wave][qi][e0] = y2[0];
        so[wave][qi][e0 + 4] = y2[1];
        if (lane == 0)
            sml[wave][qi] = make_float2(mx[qi], ls[qi]);
    }
    __syncthreads();
    // merge the waves in wave order; one (query, element) per thread and pass
    for (int t = threadIdx.x; t < QV * DH; t += VW * 64) {
        const int qi = t / DH, e = t - qi * DH;
        if (qi < Q) {
            float m = -INFINITY;
#pragma unroll
            for (int w = 0; w < VW; ++w)
                m = fmaxf(m, sml[w][qi].x);
            float L = 0.0f, O = 0.0f;
#pragma unroll
            for (int w = 0; w < VW; ++w) {
                const float2 ml = sml[w][qi];
                const float wt = (m == -INFINITY || ml.x == -INFINITY) ? 0.0f : expf(ml.x - m);
                L = fmaf(wt, ml.y, L);
                O = fmaf(wt, so[w][qi][e], O);
            }
            const int r = qi / G, head = g * G + (qi - r * G);
            const int64_t slot = ((int64_t)split * H + head) * MAX_ROWS + r;
            a.part_o[slot * DH + e] = O;
            if (e == 0)
                a.part_ml[slot] = make_float2(m, L);
        }
    }
}

// Decode attention without a combine pass: one work-group of HW waves per
// kv head, for up to QH query vectors (the draft, autoregressive and short
// verification steps of multi-head attention).  Wave w takes the 16-key
// blocks w, w + HW, ...; within a block, lane group j (16 lanes) takes keys
// j, j + 4, j + 8, j + 12 and lane e16 holds head_dim / 16 elements.  Each
// group keeps an online-softmax state; the block after next is loaded while
// the current one is used.  The groups merge by shuffles, the waves in LDS
// in wave order, and the result goes straight to the output.
constexpr int QH = 4;
constexpr int HW = 8;

template <typename TK, int ED, int NWV = HW>
__global__ __launch_bounds__(NWV * 64) void k_attn_head(AttnArgs a) {
    __shared__ float wst[NWV][QH][2];
    __shared__ float wo[NWV][QH][MAX_HEAD_DIM];
    const int g = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int pos = a.ctl->pos, M = a.ctl->m;
    if (M == 0)
        return;  // a cancelled step
    const int ctx = pos + M;
    const int dh = a.head_dim, H = a.n_heads;
    const int G = H / a.n_kv_heads;
    const int nq = G * M;  // <= QH, checked by the host
    const int ks = lane >> 4, e16 = lane & 15;
    const TK *Kg = reinterpret_cast<const TK *>(a.kcache) + (int64_t)g * a.kv_head_stride + e16 * ED;
    const TK *Vg = reinterpret_cast<const TK *>(a.vcache) + (int64_t)g * a.kv_head_stride + e16 * ED;
    const float scale = 1.0f / sqrtf((float)dh);

    float qv[QH][ED], o[QH][ED], mr[QH], lr[QH];
    int lim[QH];
#pragma unroll
    for (int qi = 0; qi < QH; ++qi) {
        mr[qi] = -INFINITY;
        lr[qi] = 0.0f;
        lim[qi] = -1;
#pragma unroll
        for (int e = 0; e < ED; ++e) {
            qv[qi][e] = 0.0f;
            o[qi][e] = 0.0f;
        }
        if (qi < nq) {
            const int r = qi / G, head = g * G + (qi - r * G);
            const float *qs = a.q + (int64_t)r * a.ld_q + (int64_t)head * dh + e16 * ED;
#pragma unroll
            for (int e = 0; e < ED; ++e)
                qv[qi][e] = qs[e] * scale;
            lim[qi] = pos + r;
        }
    }

    const int nblk = (ctx + 15) >> 4;
    KvFrag<TK, ED> kc[4], vc[4], kn[4], vn[4];
    auto load_blk = [&](int b, KvFrag<TK, ED>(&kk)[4], KvFrag<TK, ED>(&vv)[4]) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int c = b * 16 + ks + 4 * jj;
            const bool ok = b < nblk && c < ctx;
            kk[jj].load(Kg + (int64_t)(ok ? c : 0) * dh, ok);
            vv[jj].load(Vg + (int64_t)(ok ? c : 0) * dh, ok);
        }
    };
    load_blk(wave, kc, vc);
    for (int b = wave; b < nblk; b += NWV) {
        load_blk(b + NWV, kn, vn);
#pragma unroll
        for (int qi = 0; qi < QH; ++qi) {
            if (qi >= nq)
                break;
            float s[4];
            float mx = -INFINITY;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                float t = 0.0f;
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    t = fmaf(qv[qi][e], kc[jj].at(e), t);
                t += __shfl_xor(t, 1, 64);
                t += __shfl_xor(t, 2, 64);
                t += __shfl_xor(t, 4, 64);
                t += __shfl_xor(t, 8, 64);
                const int c = b * 16 + ks + 4 * jj;
                s[jj] = (c < ctx && c <= lim[qi]) ? t : -INFINITY;
                mx = fmaxf(mx, s[jj]);
            }
            const float mn = fmaxf(mr[qi], mx);
            if (mn != -INFINITY) {
                const float so = expf(mr[qi] - mn);
                float l = lr[qi] * so;
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    o[qi][e] *= so;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const float p = expf(s[jj] - mn);
                    l += p;
#pragma unroll
                    for (int e = 0; e < ED; ++e)
                        o[qi][e] = fmaf(p, vc[jj].at(e), o[qi][e]);
                }
                lr[qi] = l;
                mr[qi] = mn;
            }
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            kc[jj] = kn[jj];
            vc[jj] = vn[jj];
        }
    }
    // merge the four lane groups, then the waves
#pragma unroll
    for (int qi = 0; qi < QH; ++qi) {
        if (qi >= nq)
            break;
#pragma unroll
        for (int x = 16; x <= 32; x <<= 1) {
            const float m2 = __shfl_xor(mr[qi], x, 64), l2 = __shfl_xor(lr[qi], x, 64);
            float o2[ED];
#pragma unroll
            for (int e = 0; e < ED; ++e)
                o2[e] = __shfl_xor(o[qi][e], x, 64);
            const float mn = fmaxf(mr[qi], m2);
            if (mn != -INFINITY) {
                const float wa = expf(mr[qi] - mn), wb = expf(m2 - mn);
                lr[qi] = lr[qi] * wa + l2 * wb;
#pragma unroll
                for (int e = 0; e < ED; ++e)
                    o[qi][e] = o[qi][e] * wa + o2[e] * wb;
                mr[qi] = mn;
            }
        }
        if (ks == 0) {
#pragma unroll
            for (int e = 0; e < ED; ++e)
                wo[wave][qi][e16 * ED + e] = o[qi][e];
            if (e16 == 0) {
                wst[wave][qi][0] = mr[qi];
                wst[wave][qi][1] = lr[qi];
            }
        }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < nq * dh; t += NWV * 64) {
        const int qi = t / dh, e = t - qi * dh;
        float mx = -INFINITY;
        for (int w = 0; w < NWV; ++w)
            mx = fmaxf(mx, wst[w][qi][0]);
        float L = 0.0f, O = 0.0f;
        for (int w = 0; w < NWV; ++w) {
            const float m = wst[w][qi][0];
            if (m == -INFINITY)
                continue;
            const float wgt = expf(m - mx);
            L = fmaf(wgt, wst[w][qi][1], L);
            O = fmaf(wgt, wo[w][qi][e], O);
        }
        const int r = qi / G, head = g * G + (qi - r * G);
        const float y = O / L;
        const int64_t oi = (int64_t)r * a.ld_out + (int64_t)head * dh + e;
        if (a.out_x) {
            store_split3(a.out_x, r, head * dh + e, M, y);
        } else {
            a.out[oi] = y;
        }
    }
}

// Ordered combine of the split partials of one (head, row): deterministic.
// Thread e owns output element e.  The partial outputs of the first CB
// splits and the running maxima and sums of the first 128 are loaded before
// the control block is known: indexes are clamped to the host's bound on
// the splits, and the values of splits past the live context (stale, never
// used) are masked once the context is known.  So a context of up to CB
// chunks costs one round trip to memory (CB = 16 or 32, by the host's
// bound).  The maximum is a whole-wave max per wave; the sum of the
// rescaled split sums is a fixed tree (a wave butterfly per wave, then
// wave 0 + wave 1), so the result is the same on every run.
template <int CB>
__global__ __launch_bounds__(128) void k_attn_combine(AttnArgs a) {
    __shared__ float w_s[MAX_SPLITS];
    __shared__ float2 red[2];
    const int head = blockIdx.x, r = blockIdx.y;
    const int dh = a.head_dim, H = a.n_heads, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int S = a.splits;
    auto o_at = [&](int sp, int e) { return a.part_o[(((int64_t)sp * H + head) * MAX_ROWS + r) * dh + e]; };
    auto ml_at = [&](int sp) { return a.part_ml[((int64_t)sp * H + head) * MAX_ROWS + r]; };
    // every load of a split inside [0, S) and an element inside [0, dh)
    const int e = tid < dh ? tid : 0;
    float ov[CB];
#pragma unroll
    for (int u = 0; u < CB; ++u)
        ov[u] = o_at(min(u, S - 1), e);
    float2 ml0 = ml_at(min(tid, S - 1));
    const int pos = a.ctl->pos, M = a.ctl->m;
    if (r >= M)
        return;  // uniform over the work-group
    const int ns = (pos + M + a.chunk - 1) / a.chunk;
    if (tid >= ns)
        ml0 = make_float2(-INFINITY, 0.0f);
    float mx = ml0.x;
    for (int sp = tid + 128; sp < ns; sp += 128)
        mx = fmaxf(mx, ml_at(sp).x);
    mx = wave_max_all(mx);
    if (lane == 0)
        red[wave].x = mx;
    __syncthreads();
    mx = fmaxf(red[0].x, red[1].x);
    // split weights exp(m_s - max) and the rescaled sums, split sp by thread sp % 128
    float ls = 0.0f;
    for (int sp = tid; sp < ns; sp += 128) {
        const float2 v = sp == tid ? ml0 : ml_at(sp);
        const float w = v.x == -INFINITY ? 0.0f : expf(v.x - mx);
        w_s[sp] = w;
        ls = fmaf(w, v.y, ls);
    }
    ls = wave_sum_all(ls);
    if (lane == 0)
        red[wave].y = ls;
    __syncthreads();
    if (tid >= dh)
        return;
    const float L = red[0].y + red[1].y;
    // the splits in order: the preloaded ones, then the rest 8 at a time
    float O = 0.0f;
#pragma unroll
    for (int u = 0; u < CB; ++u)
        if (u < ns)
            O = fmaf(w_s[u], ov[u], O);
    int sp = CB;
    for (; sp + 8 <= ns; sp += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = o_at(sp + u, tid);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            O = fmaf(w_s[sp + u], v[u], O);
    }
    for (; sp < ns; ++sp)
        O = fmaf(w_s[sp], o_at(sp, tid), O);
    const float y = O / L;
    if (a.out_x) {
        store_split3(a.out_x, r, head * dh + tid, M, y);
    } else {
        a.out[(int64_t)r * a.ld_out + (int64_t)head * dh + tid] = y;
    }
}

// QB query vectors per pass: 1 or 2 when the host's bound on query vectors
// per kv head is that small (draft, autoregressive, one-draft verification
// of multi-head attention), which keeps the registers of the unused passes
// free; 4 otherwise.
template <typename TK, int QB>
static hipError_t launch_attn_split_qb(const AttnArgs &a, hipStream_t s) {
    dim3 grid(a.splits, a.n_kv_heads), block(AW * 64);
    switch (a.head_dim) {
    case 16:
        hipLaunchKernelGGL((k_attn_split<TK, 1, QB>), grid, block, 0, s, a);
        break;
    case 32:
        hipLaunchKernelGGL((k_attn_split<TK, 2, QB>), grid, block, 0, s, a);
        break;
    case 64:
        hipLaunchKernelGGL((k_attn_split<TK, 4, QB>), grid, block, 0, s, a);
        break;
    case 128:
        hipLaunchKernelGGL((k_attn_split<TK, 8, QB>), grid, block, 0, s, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipSuccess;
}

template <typename TK>
static hipError_t launch_attn_split(const AttnArgs &a, int max_q, hipStream_t s) {
    if (max_q <= 1)
        return launch_attn_split_qb<TK, 1>(a, s);
    if (max_q <= 2)
        return launch_attn_split_qb<TK, 2>(a, s);
    return launch_attn_split_qb<TK, 4>(a, s);
}

static hipError_t launch_attn_mfma(const AttnArgs &a, int max_q, hipStream_t s) {
    dim3 grid(a.splits, a.n_kv_heads, (max_q + 15) / 16), block(MW * 64);
    switch (a.head_dim) {
    case 32:
        hipLaunchKernelGGL(k_attn_mfma<32>, grid, block, 0, s, a);
        break;
    case 64:
        hipLaunchKernelGGL(k_attn_mfma<64>, grid, block, 0, s, a);
        break;
    case 128:
        hipLaunchKernelGGL(k_attn_mfma<128>, grid, block, 0, s, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipSuccess;
}

template <typename TK>
static hipError_t launch_attn_head(const AttnArgs &a, hipStream_t s) {
    dim3 grid(a.n_kv_heads), block(HW * 64);
    switch (a.head_dim) {
    case 16:
        hipLaunchKernelGGL((k_attn_head<TK, 1>), grid, block, 0, s, a);
        break;
    case 32:
        hipLaunchKernelGGL((k_attn_head<TK, 2>), grid, block, 0, s, a);
        break;
    case 64:
        hipLaunchKernelGGL((k_attn_head<TK, 4>), grid, block, 0, s, a);
        break;
    case 128:
        hipLaunchKernelGGL((k_attn_head<TK, 8>), grid, block, 0, s, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Query vectors per kv head from which bfloat16 caches take the MFMA kernel.
constexpr int ATTN_MFMA_MIN_Q = 1;

hipError_t launch_attention(const AttnArgs &a0, bool bf16, int max_rows, hipStream_t s) {
    if (a0.cap < 1 || a0.cap > MAX_CONTEXT)
        return hipErrorInvalidValue;
    AttnArgs a = a0;
    const int G = a.n_heads / a.n_kv_heads;
    const int max_q = G * max_rows;
    // one work-group per kv head while the context is short and the query
    // vectors per head fit; otherwise split the keys over work-groups
    if (max_q <= QH && a.cap <= 256)
        return bf16 ? launch_attn_head<uint16_t>(a, s) : launch_attn_head<float>(a, s);
    // (the workspace holds the partials of 64-key chunks whenever a model can
    // take this path: attn_chunk_min)
    const bool valu = bf16 && a.head_dim == 128 && max_q <= 2;
    a.chunk = valu ? ATTN_CHUNK_VALU : ATTN_CHUNK;
    a.splits = (a.cap + a.chunk - 1) / a.chunk;
    hipError_t e = hipSuccess;
    if (valu) {
        // one or two query vectors per kv head: VALU tiles
        if (max_q <= 1)
            hipLaunchKernelGGL(k_attn_valu<1>, dim3(a.splits, a.n_kv_heads), dim3(VW * 64), 0, s, a);
        else
            hipLaunchKernelGGL(k_attn_valu<2>, dim3(a.splits, a.n_kv_heads), dim3(VW * 64), 0, s, a);
    } else if (bf16 && a.head_dim >= 32 && max_q >= ATTN_MFMA_MIN_Q)
        e = launch_attn_mfma(a, max_q, s);
    else
        e = bf16 ? launch_attn_split<uint16_t>(a, max_q, s) : launch_attn_split<float>(a, max_q, s);
    if (e != hipSuccess)
        return e;
    // one work-group per (head, row) the forward can have
    if (a.splits <= 16)
        hipLaunchKernelGGL(k_attn_combine<16>, dim3(a.n_heads, max_rows), dim3(128), 0, s, a);
    else
        hipLaunchKernelGGL(k_attn_combine<32>, dim3(a.n_heads, max_rows), dim3(128), 0, s, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// small kernels

// Work-group (row r, slice b) copies elements [2048 b, 2048 b + 2048) of the
// embedding row of token r, 8 per thread with one load each, so every load
// of the row is in flight at once (d is a multiple of 8).
template <typename TW>
__global__ __launch_bounds__(256) void k_embed(const TW *E, int d, const DevCtl *ctl, float *h, int64_t ldh) {
    const int r = blockIdx.x;
    if (r >= ctl->m)
        return;
    const int i = (blockIdx.y * 256 + threadIdx.x) * 8;
    if (i >= d)
        return;
    const TW *src = E + (int64_t)ctl->tokens[r] * d + i;
    float v[8];
    if constexpr (sizeof(TW) == 2) {
        const u32x4_t w = *reinterpret_cast<const u32x4_t *>(src);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = __uint_as_float(w[j] << 16);
            v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
        }
    } else {
        const f32x4_t a = reinterpret_cast<const f32x4_t *>(src)[0];
        const f32x4_t b = reinterpret_cast<const f32x4_t *>(src)[1];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[j] = a[j];
            v[4 + j] = b[j];
        }
    }
    f32x4_t *dst = reinterpret_cast<f32x4_t *>(h + (int64_t)r * ldh + i);
    dst[0] = f32x4_t{v[0], v[1], v[2], v[3]};
    dst[1] = f32x4_t{v[4], v[5], v[6], v[7]};
}

hipError_t launch_embed(const void *emb, bool bf16, int d, const DevCtl *ctl, float *h, int64_t ldh,
                        hipStream_t s) {
    if ((d & 7) || (ldh & 7))
        return hipErrorInvalidValue;
    const dim3 grid(MAX_ROWS, (d + 2047) / 2048);
    if (bf16)
        hipLaunchKernelGGL(k_embed<uint16_t>, grid, dim3(256), 0, s, reinterpret_cast<const uint16_t *>(emb), d, ctl,
                           h, ldh);
    else
        hipLaunchKernelGGL(k_embed<float>, grid, dim3(256), 0, s, reinterpret_cast<const float *>(emb), d, ctl, h,
                           ldh);
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

// The control block from host values passed by value (no copy from host
// memory): up to MAX_ROWS tokens.
struct CtlTokens {
    int32_t t[MAX_ROWS];
};

__global__ void k_set_ctl_value(DevCtl *ctl, int32_t pos, int32_t m, CtlTokens tokens) {
    const int i = threadIdx.x;
    if (i == 0) {
        ctl->pos = pos;
        ctl->m = m;
    }
    if (i < m)
        ctl->tokens[i] = tokens.t[i];
}

hipError_t launch_set_ctl_host(DevCtl *ctl, int32_t pos, int32_t m, const int32_t *host_tokens, hipStream_t s) {
    if (m < 1 || m > MAX_ROWS)
        return hipErrorInvalidValue;
    CtlTokens t{};
    for (int i = 0; i < m; ++i)
        t.t[i] = host_tokens[i];
    hipLaunchKernelGGL(k_set_ctl_value, dim3(1), dim3(64), 0, s, ctl, pos, m, t);
    return hipGetLastError();
}

// State at the start of decoding: the cache holds the prompt minus its last
// token; the first stage drafts from that last token.
__global__ void k_init_decode(DevState *st, DevCtl *ctl, Mailbox *mb, int32_t lc, const int32_t *last,
                              int32_t max_new, int32_t k_max, ExitRule rule) {
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
    st->adaptive = rule.adaptive;
    st->gamma_d = rule.adaptive ? rule.gamma0 : (double)rule.gamma;
    st->gamma = rule.adaptive ? __double2float_rn(rule.gamma0) : rule.gamma;
    st->n_updates = 0;
    st->ar = 0.0;
    st->alpha = rule.alpha;
    st->epsilon = rule.epsilon;
    st->beta1 = rule.beta1;
    st->beta2 = rule.beta2;
    st->n_stages = st->n_drafted = st->n_accepted = st->n_draft_steps = 0;
    ctl->pos = lc;
    ctl->m = 1;
    ctl->m_next = 1;
    ctl->tokens[0] = tok;
    if (mb)
        __hip_atomic_store(&mb->word, mb_pack(0, st->phase, st->gen_done, 0), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_SYSTEM);
}

hipError_t launch_init_decode(DevState *st, DevCtl *ctl, Mailbox *mb, int32_t lc, const int32_t *dev_last,
                              int32_t max_new, int32_t k_max, const ExitRule &rule, hipStream_t s) {
    hipLaunchKernelGGL(k_init_decode, dim3(1), dim3(64), 0, s, st, ctl, mb, lc, dev_last, max_new, k_max, rule);
    return hipGetLastError();
}

__global__ void k_step_guard(DevCtl *ctl, const DevState *st, int32_t phase, int32_t max_rows) {
    if (threadIdx.x != 0)
        return;
    // the host and the device agree on a step's kind and rows exactly
    const int mn = ctl->m_next;
    const bool ok = !st->gen_done && st->phase == phase && mn == max_rows;
    ctl->m = ok ? mn : 0;
}

hipError_t launch_step_guard(DevCtl *ctl, const DevState *st, int32_t phase, int32_t max_rows, hipStream_t s) {
    if (max_rows < 1 || max_rows > MAX_ROWS)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_step_guard, dim3(1), dim3(64), 0, s, ctl, st, phase, max_rows);
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
