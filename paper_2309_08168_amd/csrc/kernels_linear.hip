// Weight-streaming linear layers of the decoder forward, with their fused
// prologue (RMSNorm) and epilogues (rotary embedding + KV append, SwiGLU,
// residual add, greedy head with the draft-exit test and acceptance).
//
// Every step of greedy decoding at batch 1 streams the whole weight set
// once (Sec. 3.1: model size over memory bandwidth bounds the decode
// speed), so the main loops below are built to read each weight byte
// exactly once with 16-byte loads:
//   - k_linear_valu, MR == 1: the GEMV of a draft or autoregressive step;
//   - k_linear_valu, MR == 2: verification of one draft (one-wave tiles for
//     bf16 weights);
//   - k_linear_valu, MR == 16: any row count, for float32 weights;
//   - k_linear_mfma: the verification forward over up to 16 rows (the last
//     committed token plus the drafts, Algorithm 2) on bf16 MFMA tiles, the
//     activations split into three bf16 terms packed into the 16 columns.
//
// RMSNorm is folded in: y = W (g * h) / rms(h), so the kernel that reads h
// as its input also accumulates sum(h^2) and scales its outputs at the end;
// no separate normalisation pass.
#include <hip/hip_ext.h>

#include "sd_internal.h"
#include "decode_step.h"

namespace sdk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8_t __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float32 -> bfloat16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void unpack8(u32x4_t v, float (&w)[8]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        w[2 * j] = __uint_as_float(v[j] << 16);
        w[2 * j + 1] = __uint_as_float(v[j] & 0xffff0000u);
    }
}

// Weights are read once per step: non-temporal loads keep them from
// displacing the activations and KV in the caches.
__device__ __forceinline__ void ldw8(const uint16_t *p, float (&w)[8]) {
    unpack8(__builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p)), w);
}
__device__ __forceinline__ void ldw8(const float *p, float (&w)[8]) {
    f32x4_t a = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p));
    f32x4_t b = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p) + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        w[j] = a[j];
        w[4 + j] = b[j];
    }
}
__device__ __forceinline__ void ldg8(const uint16_t *p, float (&w)[8]) {
    unpack8(*reinterpret_cast<const u32x4_t *>(p), w);
}
__device__ __forceinline__ void ldg8(const float *p, float (&w)[8]) {
    f32x4_t a = reinterpret_cast<const f32x4_t *>(p)[0];
    f32x4_t b = reinterpret_cast<const f32x4_t *>(p)[1];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        w[j] = a[j];
        w[4 + j] = b[j];
    }
}

__device__ __forceinline__ void store_kv(float *p, float v) { *p = v; }
__device__ __forceinline__ void store_kv(uint16_t *p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, 64);
    return v;
}

// ---------------------------------------------------------------------------
// Which weight rows a tile of R rows covers.
//   QKV: R/2 rotary pairs (i, i + head_dim/2) of one head, so the epilogue
//        can rotate q and k in place;
//   SWIGLU: R/2 gate rows and the R/2 matching up rows;
//   otherwise R consecutive rows.

template <int EPI>
__device__ __forceinline__ int tile_row(int t, int i, int R, const EpiArgs &e) {
    if constexpr (EPI == EPI_QKV) {
        const int P = R >> 1, half = e.head_dim >> 1, per_head = half / P;
        const int head = t / per_head, p0 = (t - head * per_head) * P;
        return head * e.head_dim + (i < P ? p0 + i : half + p0 + (i - P));
    } else if constexpr (EPI == EPI_SWIGLU) {
        const int P = R >> 1;
        return i < P ? t * P + i : e.ffn + t * P + (i - P);
    } else {
        return t * R + i;
    }
}

template <int EPI>
__device__ __forceinline__ bool row_valid(int t, int i, int R, int N, const EpiArgs &e) {
    if constexpr (EPI == EPI_QKV) {
        return true;
    } else if constexpr (EPI == EPI_SWIGLU) {
        const int P = R >> 1;
        return t * P + (i < P ? i : i - P) < e.ffn;
    } else {
        return t * R + i < N;
    }
}

// ---------------------------------------------------------------------------
// Greedy head: argmax and top-1 probability across all tiles.

struct HeadPart {
    float mx;
    int idx;
    float sum;  // sum over the part of exp(l - mx)
};

__device__ __forceinline__ HeadPart head_empty() { return HeadPart{-INFINITY, 0x7fffffff, 0.0f}; }

__device__ __forceinline__ HeadPart head_comb(HeadPart a, HeadPart b) {
    if (b.sum == 0.0f)
        return a;
    if (a.sum == 0.0f)
        return b;
    const float mx = fmaxf(a.mx, b.mx);
    HeadPart r;
    r.mx = mx;
    r.idx = (b.mx > a.mx || (b.mx == a.mx && b.idx < a.idx)) ? b.idx : a.idx;
    r.sum = a.sum * expf(a.mx - mx) + b.sum * expf(b.mx - mx);
    return r;
}

// The decoding decision after one step, taken by one thread once the
// argmax y[r] and top-1 probability p[r] of every row are known.
//   AR:     Algorithm 1, append y and feed it back.
//   DRAFT:  Algorithm 2 drafting with the exit of Sec. 3.4: keep d_j, stop
//           after it when p_j < gamma or the stage budget is reached.
//   VERIFY: Algorithm 2 verification: the longest prefix of drafts equal
//           to the model's own tokens is accepted, followed by the model's
//           token at the first mismatch (or the bonus token).
// The state updates themselves are shared with the sampling variant.
__device__ void decode_decision(const HeadArgs &h, DevCtl *ctl, const int *y, const float *p) {
    DevState *st = h.st;
    if (h.mode == HEAD_AR) {
        ar_commit(h, ctl, y[0]);
    } else if (h.mode == HEAD_DRAFT) {
        draft_commit(h, ctl, y[0], p[0]);
    } else if (h.mode == HEAD_VERIFY) {
        int n = 0;
        while (n < st->k && st->drafts[n] == y[n])
            ++n;
        stage_commit(h, ctl, n, y[n]);
    }
}

// One work-group after the head: combine the per-tile partials of every
// row in a fixed order (deterministic), then take the decoding decision.
// Thread j takes tiles j, j + 256, ... of every row; the loads of up to
// HF_BATCH tiles per thread are issued together (one round trip for up to
// 4096 tiles), then the 256 partial results of a row are combined by a
// fixed tree across lanes and waves.
__device__ HeadPart head_shfl(HeadPart v, int o) {
    HeadPart r;
    r.mx = __shfl_xor(v.mx, o, 64);
    r.idx = __shfl_xor(v.idx, o, 64);
    r.sum = __shfl_xor(v.sum, o, 64);
    return r;
}

constexpr int HF_THREADS = 256;
constexpr int HF_BATCH = 16;

__device__ void head_finalize(const LinearArgs &a, int n_tiles, int M) {
    constexpr int NWF = HF_THREADS / 64;
    __shared__ HeadPart wred[NWF][MAX_ROWS];
    __shared__ int ys[MAX_ROWS];
    __shared__ float ps[MAX_ROWS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const HeadArgs &h = a.epi.head;
    for (int m = 0; m < M; ++m) {
        HeadPart acc = head_empty();
        for (int t0 = 0; t0 < n_tiles; t0 += HF_THREADS * HF_BATCH) {
            // tiles past n_tiles read the last one and are skipped
            float4 v[HF_BATCH];
#pragma unroll
            for (int u = 0; u < HF_BATCH; ++u)
                v[u] = h.partials[(int64_t)min(t0 + tid + HF_THREADS * u, n_tiles - 1) * MAX_ROWS + m];
#pragma unroll
            for (int u = 0; u < HF_BATCH; ++u)
                if (t0 + tid + HF_THREADS * u < n_tiles)
                    acc = head_comb(acc, HeadPart{v[u].x, __float_as_int(v[u].y), v[u].z});
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1)
            acc = head_comb(acc, head_shfl(acc, o));
        if (lane == 0)
            wred[wave][m] = acc;
    }
    __syncthreads();
    if (tid < M) {
        HeadPart r = wred[0][tid];
        for (int w = 1; w < NWF; ++w)
            r = head_comb(r, wred[w][tid]);
        ys[tid] = r.idx;
        ps[tid] = 1.0f / r.sum;
    }
    __syncthreads();
    if (tid == 0)
        decode_decision(h, const_cast<DevCtl *>(a.ctl), ys, ps);
}

// ---------------------------------------------------------------------------
// Epilogues.  fin[i * MR + m] holds the raw dot product of tile row i and
// input row m; inv[m] the RMSNorm scale of row m (1 without a norm).

// The residual-stream value an output projection adds to does not depend
// on the products: the VALU kernels load it before their main loop, so the
// round trip overlaps the loop instead of ending the kernel.  Thread j loads
// what epilogue element j needs (R * MR is at most the work-group size);
// indexes are clamped, so rows past the forward's row count read valid
// memory that is never used.  (Loading the QKV tile's rotary factors the same
// way made the one-row layer slower: their address waits for the control
// block's position before the first weight load.)
struct EpiPre {
    float res;
    bool ok;
};

template <int EPI>
__device__ __forceinline__ EpiPre epi_prefetch(const LinearArgs &a, int t, int R, int MR) {
    EpiPre p{0.0f, false};
    if constexpr (EPI == EPI_RESID) {
        const EpiArgs &e = a.epi;
        const int j = min((int)threadIdx.x, R * MR - 1);
        const int i = j % R, m = j / R;
        const int n = min(t * R + i, a.N - 1);
        p.res = e.out[(int64_t)m * e.ld_out + n];
        p.ok = true;
    }
    return p;
}

template <typename TK, int EPI>
__device__ __forceinline__ void run_epilogue(const LinearArgs &a, float *fin, int R, int MR, const float *inv, int t,
                                             int M, const EpiPre &pre = EpiPre{0.0f, false}) {
    const int tid = threadIdx.x;
    const EpiArgs &e = a.epi;
    if constexpr (EPI == EPI_PARTIAL) {
        float *dst = a.part + (int64_t)(blockIdx.x % a.splits) * MAX_ROWS * a.N;
        for (int j = tid; j < R * M; j += blockDim.x) {
            const int i = j % R, m = j / R, n = t * R + i;
            if (n < a.N)
                dst[(int64_t)m * a.N + n] = fin[i * MR + m];
        }
    } else if constexpr (EPI == EPI_STORE || EPI == EPI_RESID) {
        for (int j = tid; j < R * M; j += blockDim.x) {
            const int i = j % R, m = j / R, n = t * R + i;
            if (n < a.N) {
                const float v = fin[i * MR + m] * inv[m];
                float *o = e.out + (int64_t)m * e.ld_out + n;
                if constexpr (EPI == EPI_RESID) {
                    *o = (pre.ok && j == tid ? pre.res : *o) + v;
                } else {
                    *o = v;
                }
            }
        }
    } else if constexpr (EPI == EPI_SWIGLU) {
        const int P = R >> 1;
        for (int j = tid; j < P * M; j += blockDim.x) {
            const int i = j % P, m = j / P, f = t * P + i;
            if (f < e.ffn) {
                const float g = fin[i * MR + m] * inv[m];
                const float u = fin[(i + P) * MR + m] * inv[m];
                const float y = g / (1.0f + expf(-g)) * u;
                if (e.out_x) {
                    store_split3(e.out_x, m, f, M, y);
                } else {
                    e.out[(int64_t)m * e.ld_out + f] = y;
                }
            }
        }
    } else if constexpr (EPI == EPI_QKV) {
        const int P = R >> 1, dh = e.head_dim, half = dh >> 1;
        const int H = e.n_heads, KVH = e.n_kv_heads;
        for (int j = tid; j < P * M; j += blockDim.x) {
            const int i = j % P, m = j / P;
            const int n0 = tile_row<EPI>(t, i, R, e);
            const int head = n0 / dh, ei = n0 - head * dh;
            float y0 = fin[i * MR + m] * inv[m];
            float y1 = fin[(i + P) * MR + m] * inv[m];
            const int pos = a.ctl->pos + m;
            if (head < H + KVH) {
                const float2 cs = e.rope[(int64_t)pos * half + ei];
                const float r0 = y0 * cs.x - y1 * cs.y;
                const float r1 = y1 * cs.x + y0 * cs.y;
                y0 = r0;
                y1 = r1;
            }
            if (head < H) {
                float *q = e.q + (int64_t)m * e.ld_q + (int64_t)head * dh + ei;
                q[0] = y0;
                q[half] = y1;
            } else {
                const bool is_k = head < H + KVH;
                const int g = is_k ? head - H : head - H - KVH;
                TK *base = reinterpret_cast<TK *>(is_k ? e.kcache : e.vcache) + (int64_t)g * e.kv_head_stride +
                           (int64_t)pos * dh + ei;
                store_kv(base, y0);
                store_kv(base + half, y1);
            }
        }
    } else if constexpr (EPI == EPI_HEAD) {
        const HeadArgs &h = e.head;
        for (int j = tid; j < R * M; j += blockDim.x) {
            const int i = j % R, m = j / R, n = t * R + i;
            if (n < a.N) {
                const float v = fin[i * MR + m] * inv[m];
                fin[i * MR + m] = v;
                if (h.logits)
                    h.logits[(int64_t)(h.logits_by_draft ? h.st->k : m) * h.ld_logits + n] = v;
            }
        }
        __syncthreads();
        if (tid < M) {
            const int m = tid;
            float mx = -INFINITY;
            int ix = 0x7fffffff;
            for (int i = 0; i < R && t * R + i < a.N; ++i) {
                const float v = fin[i * MR + m];
                if (v > mx) {
                    mx = v;
                    ix = t * R + i;
                }
            }
            float s = 0.0f;
            for (int i = 0; i < R && t * R + i < a.N; ++i)
                s += expf(fin[i * MR + m] - mx);
            h.partials[(int64_t)t * MAX_ROWS + m] = make_float4(mx, __int_as_float(ix), s, 0.0f);
        }
        __syncthreads();
    }
}

// One work-group after the head: combine the partials of all tiles and take
// the decoding decision.
__global__ __launch_bounds__(HF_THREADS) void k_head_finalize(LinearArgs a) {
    const int M = a.ctl->m;
    if (M == 0)
        return;  // a cancelled step takes no decision
    head_finalize(a, a.n_tiles, M);
}

// ---------------------------------------------------------------------------
// VALU main loop: one work-group per tile of R weight rows; the NT threads
// stride over the reduction dimension in chunks of 8 elements (one 16-byte
// load of bf16 weights per row), then reduce across the work-group.  MR is
// the largest row count handled (1: the GEMV).
//
// NT = 256: four waves share a tile and meet in LDS.  NT = 64: one wave
// owns its tile over the whole reduction (bf16 weights, up to 4 rows), so
// the reduction is a wave sum with no cross-wave step, and the loads of U
// chunks are issued before the first is used.  Measured at the 13B shapes,
// the one-wave tiles are the faster choice for every layer at two rows
// (down 27.8 -> 25.6 us, O 13.0 -> 11.8 us); at one row the four-wave
// tiles are as fast or faster.  Keeping the next chunk's loads in flight
// while the current one is used (software pipelining) was slower at every
// shape: the extra registers cost more occupancy than the overlap gained.

template <typename TW, int MR, int R, int EPI, bool NORM, int NT = 256, int U = 1>
__global__ __launch_bounds__(NT) void k_linear_valu(LinearArgs a) {
    static_assert(NT == 256 || NT == 64, "four-wave or one-wave tiles");
    static_assert(NT == 256 || (sizeof(TW) == 2 && MR <= 4), "one-wave tiles take bf16 weights and up to 4 rows");
    constexpr int NWAVE = NT / 64;
    constexpr int NV = MR * R + (NORM ? MR : 0);
    __shared__ float red[NWAVE][NV];
    __shared__ float fin[R * MR];
    __shared__ float inv_s[MR];
    const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int M = MR == 1 ? 1 : a.ctl->m;
    const EpiPre pre = epi_prefetch<EPI>(a, t, R, MR);
    const int K = a.K, nch = K >> 3;
    const TW *W = reinterpret_cast<const TW *>(a.W);
    const TW *G = reinterpret_cast<const TW *>(a.gain);

    int64_t roff[R];
#pragma unroll
    for (int i = 0; i < R; ++i)
        roff[i] = row_valid<EPI>(t, i, R, a.N, a.epi) ? (int64_t)tile_row<EPI>(t, i, R, a.epi) * K : 0;

    float acc[MR][R];
    float ss[MR];
#pragma unroll
    for (int r = 0; r < MR; ++r) {
        ss[r] = 0.0f;
#pragma unroll
        for (int i = 0; i < R; ++i)
            acc[r][i] = 0.0f;
    }

    // Up to 4 rows, every row's product is computed, whatever the row count
    // (the X buffers hold MAX_ROWS rows; rows past M are never stored), and
    // the weight, gain and X loads of an iteration are all issued before the
    // first is used: a branch around the X loads, or unpacking as loads
    // arrive, would make the compiler wait for each group of loads in turn.
    constexpr bool BATCH = MR > 1 && MR <= 4 && sizeof(TW) == 2;
    if constexpr (NT == 64) {
        auto issue = [&](int c, u32x4_t(&wr)[R], u32x4_t &gr, f32x4_t(&xr)[MR][2]) {
#pragma unroll
            for (int i = 0; i < R; ++i)
                wr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(W + roff[i] + (int64_t)c * 8));
            if constexpr (NORM)
                gr = *reinterpret_cast<const u32x4_t *>(G + c * 8);
            else
                gr = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
            for (int r = 0; r < MR; ++r) {
                xr[r][0] = reinterpret_cast<const f32x4_t *>(a.X + (int64_t)r * a.ldx + c * 8)[0];
                xr[r][1] = reinterpret_cast<const f32x4_t *>(a.X + (int64_t)r * a.ldx + c * 8)[1];
            }
        };
        auto use = [&](const u32x4_t(&wr)[R], const u32x4_t &gr, const f32x4_t(&xr)[MR][2]) {
            float g[8], w[R][8];
            if constexpr (NORM)
                unpack8(gr, g);
#pragma unroll
            for (int i = 0; i < R; ++i)
                unpack8(wr[i], w[i]);
#pragma unroll
            for (int r = 0; r < MR; ++r) {
                float x[8];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    x[k] = xr[r][0][k];
                    x[4 + k] = xr[r][1][k];
                }
                if constexpr (NORM) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        ss[r] = fmaf(x[k], x[k], ss[r]);
                        x[k] *= g[k];
                    }
                }
#pragma unroll
                for (int i = 0; i < R; ++i)
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        acc[r][i] = fmaf(w[i][k], x[k], acc[r][i]);
            }
        };
        int c = tid;
        for (; c + 64 * (U - 1) < nch; c += 64 * U) {
            u32x4_t wr[U][R], gr[U];
            f32x4_t xr[U][MR][2];
#pragma unroll
            for (int u = 0; u < U; ++u)
                issue(c + 64 * u, wr[u], gr[u], xr[u]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < U; ++u)
                use(wr[u], gr[u], xr[u]);
        }
        if constexpr (U > 1) {
            for (; c < nch; c += 64) {
                u32x4_t wr[R], gr;
                f32x4_t xr[MR][2];
                issue(c, wr, gr, xr);
                __builtin_amdgcn_sched_barrier(0);
                use(wr, gr, xr);
            }
        }
    } else
    for (int c = tid; c < nch; c += 256) {
        float w[R][8];
        float g[8];
        float xb[BATCH ? MR : 1][8];
        if constexpr (BATCH) {
            u32x4_t wr[R], gr;
#pragma unroll
            for (int i = 0; i < R; ++i)
                wr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(W + roff[i] + (int64_t)c * 8));
            if constexpr (NORM)
                gr = *reinterpret_cast<const u32x4_t *>(G + c * 8);
            f32x4_t xr[MR][2];
#pragma unroll
            for (int r = 0; r < MR; ++r) {
                xr[r][0] = reinterpret_cast<const f32x4_t *>(a.X + (int64_t)r * a.ldx + c * 8)[0];
                xr[r][1] = reinterpret_cast<const f32x4_t *>(a.X + (int64_t)r * a.ldx + c * 8)[1];
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < R; ++i)
                unpack8(wr[i], w[i]);
            if constexpr (NORM)
                unpack8(gr, g);
#pragma unroll
            for (int r = 0; r < MR; ++r)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    xb[r][k] = xr[r][0][k];
                    xb[r][4 + k] = xr[r][1][k];
                }
        } else {
#pragma unroll
            for (int i = 0; i < R; ++i)
                ldw8(W + roff[i] + (int64_t)c * 8, w[i]);
            if constexpr (NORM)
                ldg8(G + c * 8, g);
        }
#pragma unroll
        for (int r = 0; r < MR; ++r) {
            if (BATCH || r < M) {
                float x[8];
                if constexpr (BATCH) {
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        x[k] = xb[r][k];
                } else {
                    ldg8(a.X + (int64_t)r * a.ldx + c * 8, x);
                }
                if constexpr (NORM) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        ss[r] = fmaf(x[k], x[k], ss[r]);
                        x[k] *= g[k];
                    }
                }
#pragma unroll
                for (int i = 0; i < R; ++i)
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        acc[r][i] = fmaf(w[i][k], x[k], acc[r][i]);
            }
        }
    }

    // wave sums of every row's products (rows past M too: their values are
    // never used) and of the sums of squares, up to 16 at a time
    {
        constexpr int NA = MR * R, NC = NA < 16 ? NA : 16;
        static_assert((NA & (NA - 1)) == 0, "a power of two of products per lane");
        const int j = wave_sums_index(lane) & (NC - 1);
        const bool owner = lane == wave_sums_lane(j);
#pragma unroll
        for (int c0 = 0; c0 < NA; c0 += NC) {
            float part[NC];
#pragma unroll
            for (int u = 0; u < NC; ++u)
                part[u] = acc[(c0 + u) / R][(c0 + u) % R];
            const float v = wave_sums<NC>(part, lane);
            if (owner)
                red[wave][c0 + j] = v;
        }
        if constexpr (NORM) {
            constexpr int NS = MR < 16 ? MR : 16;
            const int js = wave_sums_index(lane) & (NS - 1);
#pragma unroll
            for (int c0 = 0; c0 < MR; c0 += NS) {
                float part[NS];
#pragma unroll
                for (int u = 0; u < NS; ++u)
                    part[u] = ss[c0 + u];
                const float v = wave_sums<NS>(part, lane);
                if (lane == wave_sums_lane(js))
                    red[wave][MR * R + c0 + js] = v;
            }
        }
    }
    __syncthreads();
    auto waves_sum = [&](int j) {
        if constexpr (NWAVE == 1)
            return red[0][j];
        else
            return (red[0][j] + red[1][j]) + (red[2][j] + red[3][j]);
    };
    for (int j = tid; j < MR * R; j += NT) {
        const int r = j / R, i = j - r * R;
        if (r < M)
            fin[i * MR + r] = waves_sum(j);
    }
    if (tid < MR) {
        float v = 1.0f;
        if constexpr (NORM) {
            if (tid < M)
                v = 1.0f / sqrtf(waves_sum(MR * R + tid) / (float)K + a.eps);
        }
        inv_s[tid] = v;
    }
    __syncthreads();
    // A cancelled step (ctl->m = 0) streams its weights and writes nothing.
    // The one-row path reads ctl->m only here and only when the launch may
    // be cancelled: a branch on it before the first loads delays every
    // launch.
    run_epilogue<TW, EPI>(a, fin, R, MR, inv_s, t, (MR == 1 && a.guarded) ? a.ctl->m : M, pre);
}

// ---------------------------------------------------------------------------
// FP8 draft weights.  The adaptation appendix runs self-speculative decoding
// on FP8 and FP4 weights; here a copy of the draft's weights is quantized so
// that a draft step streams one byte per weight, while verification keeps
// the stored bf16 weights (the output stays exactly greedy bf16 decoding).
// Format: OCP FP8 E4M3 (bias 7, largest value 448, S.1111.111 NaN) with one
// power-of-two scale 2^e per output row, e the smallest integer with
// max|W[n][:]| 2^-e <= 448; the byte is the nearest E4M3 value (ties to
// even) of W[n][k] 2^-e.  Scaling by 2^-e is exact, so every step is.

// The E4M3 byte of v, |v| <= 448, to nearest with ties to even.
__device__ __forceinline__ uint32_t fp8_encode(float v) {
    const uint32_t sgn = (__float_as_uint(v) >> 24) & 0x80u;
    const float a = fabsf(v);
    if (a == 0.0f)
        return sgn;
    int e;
    (void)frexpf(a, &e);  // a = f 2^e, 0.5 <= f < 1
    const int quantum = e - 1 < -6 ? -9 : e - 4;
    const float r = ldexpf(rintf(ldexpf(a, -quantum)), quantum);  // rintf: ties to even
    if (r == 0.0f)
        return sgn;
    (void)frexpf(r, &e);
    const int ex = e - 1;
    if (ex < -6)
        return sgn | (uint32_t)ldexpf(r, 9);
    return sgn | (uint32_t)((ex + 7) << 3) | (uint32_t)(ldexpf(r, -ex) * 8.0f - 8.0f);
}

// One work-group per row: the row's largest magnitude, its exponent, then
// the bytes.
__global__ __launch_bounds__(256) void k_quantize_fp8(const uint16_t *W, int32_t K, uint8_t *Q, int32_t *E) {
    __shared__ float red[4];
    const int64_t n = blockIdx.x;
    const uint16_t *w = W + n * K;
    float amax = 0.0f;
    for (int k = threadIdx.x; k < K; k += 256)
        amax = fmaxf(amax, fabsf(bf2f(w[k])));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, o, 64));
    if ((threadIdx.x & 63) == 0)
        red[threadIdx.x >> 6] = amax;
    __syncthreads();
    amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    int e = 0;
    if (amax > 0.0f) {
        int ea;
        const float f = frexpf(amax, &ea);  // amax = f 2^ea; 448 = 0.875 2^9
        e = ea - 9 + (f > 0.875f ? 1 : 0);
    }
    if (threadIdx.x == 0)
        E[n] = e;
    for (int k = threadIdx.x; k < K; k += 256)
        Q[n * K + k] = (uint8_t)fp8_encode(ldexpf(bf2f(w[k]), -e));
}

hipError_t launch_quantize_fp8(const uint16_t *W, int32_t N, int32_t K, uint8_t *Q, int32_t *E, hipStream_t s) {
    if (N < 1 || K < 1)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_quantize_fp8, dim3(N), dim3(256), 0, s, W, K, Q, E);
    return hipGetLastError();
}

// One-row GEMV over FP8 weights (draft steps): a tile of R weight rows per
// work-group of FP8_WAVES waves; each thread takes 16 consecutive elements
// of the reduction per step, one 16-byte load per weight row, converted to
// float32 exactly by the hardware.  RMSNorm is folded in as in
// k_linear_valu; the row's 2^e scales its dot product before the shared
// epilogues.
// Measured at the 13B shapes (cold weights, kernel time): two waves per
// tile against four, QKV 17.2 against 18.1 us, O 7.3 against 7.9, gate/up
// 26.8 against 26.6, down 14.6 against 15.5; one wave loses on the narrow
// layers, 16-row tiles and a software-pipelined loop lose everywhere, and
// a decode through fp16 bits is slower than the conversion instruction.
// Against a plain read of the same bytes (gate/up 21.1 us), the activation
// and gain loads cost about 2 us and the arithmetic that does not overlap
// the loads about 2 us more.
typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr int FP8_WAVES = 2;

template <int R, int EPI, bool NORM>
__global__ __launch_bounds__(FP8_WAVES * 64) void k_linear_fp8(LinearArgs a) {
    constexpr int NT = FP8_WAVES * 64;
    constexpr int NV = R + (NORM ? 1 : 0);
    __shared__ float red[FP8_WAVES][NV];
    __shared__ float fin[R];
    __shared__ float inv_s[1];
    const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int K = a.K, nch = K >> 4;
    const uint8_t *W = reinterpret_cast<const uint8_t *>(a.W);
    const uint16_t *G = reinterpret_cast<const uint16_t *>(a.gain);
    int rows[R];
    int64_t roff[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        rows[i] = row_valid<EPI>(t, i, R, a.N, a.epi) ? tile_row<EPI>(t, i, R, a.epi) : 0;
        roff[i] = (int64_t)rows[i] * K;
    }
    // the row exponent and the residual value the epilogue needs, in flight during the loop
    const int wexp = a.wexp[rows[min(tid, R - 1)]];
    const EpiPre pre = epi_prefetch<EPI>(a, t, R, 1);
    float acc[R], ss = 0.0f;
#pragma unroll
    for (int i = 0; i < R; ++i)
        acc[i] = 0.0f;
    for (int c = tid; c < nch; c += NT) {
        u32x4_t wr[R], gr[2];
        f32x4_t xr[4];
#pragma unroll
        for (int i = 0; i < R; ++i)
            wr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(W + roff[i] + (int64_t)c * 16));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            xr[j] = reinterpret_cast<const f32x4_t *>(a.X + (int64_t)c * 16)[j];
        if constexpr (NORM) {
            gr[0] = reinterpret_cast<const u32x4_t *>(G + c * 16)[0];
            gr[1] = reinterpret_cast<const u32x4_t *>(G + c * 16)[1];
        }
        __builtin_amdgcn_sched_barrier(0);
        float x[16];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int k = 0; k < 4; ++k)
                x[4 * j + k] = xr[j][k];
        if constexpr (NORM) {
            float g[2][8];
            unpack8(gr[0], g[0]);
            unpack8(gr[1], g[1]);
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                ss = fmaf(x[k], x[k], ss);
                x[k] *= g[k >> 3][k & 7];
            }
        }
#pragma unroll
        for (int i = 0; i < R; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x2_t lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)wr[i][j], false);
                const f32x2_t hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)wr[i][j], true);
                acc[i] = fmaf(lo[0], x[4 * j], acc[i]);
                acc[i] = fmaf(lo[1], x[4 * j + 1], acc[i]);
                acc[i] = fmaf(hi[0], x[4 * j + 2], acc[i]);
                acc[i] = fmaf(hi[1], x[4 * j + 3], acc[i]);
            }
    }
    {
        const int j = wave_sums_index(lane) & (R - 1);
        const float v = wave_sums<R>(acc, lane);
        if (lane == wave_sums_lane(j))
            red[wave][j] = v;
        if constexpr (NORM) {
            const float s = wave_sums<1>({ss}, lane);
            if (lane == 0)
                red[wave][R] = s;
        }
    }
    __syncthreads();
    auto waves_sum = [&](int j) {
        float v = red[0][j];
#pragma unroll
        for (int w = 1; w < FP8_WAVES; ++w)
            v += red[w][j];
        return v;
    };
    if (tid < R)
        fin[tid] = ldexpf(waves_sum(tid), wexp);
    if (tid == 0)
        inv_s[0] = NORM ? 1.0f / sqrtf(waves_sum(R) / (float)K + a.eps) : 1.0f;
    __syncthreads();
    // a cancelled step (ctl->m = 0) writes nothing; see k_linear_valu
    run_epilogue<uint16_t, EPI>(a, fin, R, 1, inv_s, t, a.guarded ? a.ctl->m : 1, pre);
}

template <int R>
static hipError_t launch_fp8_r(const LinearArgs &a, int epi, int n_tiles, hipStream_t s, const LaunchTiming &t) {
    dim3 grid(n_tiles), block(FP8_WAVES * 64);
    switch (epi) {
    case EPI_RESID:
        launch_k(k_linear_fp8<R, EPI_RESID, false>, grid, block, s, t, a);
        break;
    case EPI_SWIGLU:
        launch_k(k_linear_fp8<R, EPI_SWIGLU, true>, grid, block, s, t, a);
        break;
    case EPI_QKV:
        launch_k(k_linear_fp8<R, EPI_QKV, true>, grid, block, s, t, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// MFMA main loop (bf16 weights, up to 16 rows).  A work-group owns TN tiles
// of 16 weight rows and the whole reduction dimension (or one of S slices of
// it); its NW waves take every NW-th 128-element k-step, so at any time the
// work-group reads adjacent pieces of its rows, and are summed in LDS at the
// end: no work-group depends on another.
//
// The MFMA operand layout puts weight row l % 16 in lane l, so loading it
// straight from memory gives every lane its own cache line and defeats the
// coalescing of neighbouring lanes (one L1 access per lane instead of one
// per four).  Weights are therefore loaded coalesced (16 lanes per 256-byte
// row slice), non-temporal (they are read once), and transposed through a
// wave-private LDS tile whose 16-byte chunks are XOR-swizzled by row, which
// keeps both the writes and the fragment reads free of bank conflicts.
// The activations come pre-split (three bf16 terms) in fragment order
// (xfrag_off), so each B operand is one contiguous 1 KB load.  A k-step is
// four 16x16x32 MFMAs per tile and packing; the k order inside an MFMA is a
// permutation shared by both operands, so the dot products are unchanged.

// The 16 x NP columns of the B operand hold (term, row) pairs: column
// c = t * M + r carries term t of activation row r, so NP = ceil(3 M / 16)
// MFMAs per k-step cover all X_TERMS terms of M rows (one MFMA for up to 5
// rows, two up to 10, three up to 16).  The host picks NP from its bound on
// M (LinearArgs::max_rows).
//
// The launch bound asks for two waves per SIMD up to four tiles (eight do
// not fit twice in LDS or in the registers).  With one set of activation
// registers (below) the four-tile kernel at three packings fits that in 218
// registers without spilling; double-buffered activations took 260 (one
// wave per SIMD), and 13B verification at 13-16 rows was 2% slower.
template <int EPI, int TN, int NW, int NP>
__global__ __launch_bounds__(NW * 64, TN <= 4 ? 2 : 1) void k_linear_mfma(LinearArgs a) {
    constexpr int WL = TN * 16 * 128;                // bf16 staging per wave
    constexpr int RC = NP * 16 + 1;                  // reduction row length
    constexpr size_t SMEM_W = (size_t)NW * WL * 2, SMEM_R = (size_t)NW * TN * 16 * RC * 4;
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM_W > SMEM_R ? SMEM_W : SMEM_R];
    __shared__ float fin[TN * 16 * 16];
    __shared__ float inv_s[16];
    const int S = EPI == EPI_PARTIAL ? a.splits : 1;
    const int grp = blockIdx.x / S, sp = blockIdx.x - grp * S;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r16 = lane & 15, kg = lane >> 4;
    const int M = a.ctl->m;  // 0 in a cancelled step: nothing is written
    const int n_tiles = a.n_tiles;
    uint16_t *wl = reinterpret_cast<uint16_t *>(smem) + wave * WL;
    // coalesced loads: instruction ii of tile j reads rows 4 ii + lane / 16,
    // 16-byte chunk lane % 16 of the k-step's 256-byte slice
    const int lrow = lane >> 4, lch = lane & 15;
    uint32_t woff[TN][4];
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
            const int t = grp * TN + j, row = 4 * ii + lrow;
            const bool nv = t < n_tiles && row_valid<EPI>(t, row, 16, a.N, a.epi);
            woff[j][ii] = (uint32_t)(nv ? tile_row<EPI>(t, row, 16, a.epi) : 0) * (uint32_t)a.K + lch * 8;
        }
    const uint16_t *W = reinterpret_cast<const uint16_t *>(a.W);
    const uint16_t *X = a.Xs + lane * 8;
    // k-steps of this split, dealt out to the waves in turn
    const int KS_all = a.K >> 7;
    const int ks0 = (int)(((int64_t)KS_all * sp) / S), ks1 = (int)(((int64_t)KS_all * (sp + 1)) / S);

    floatx4_t acc[TN][NP];
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int p = 0; p < NP; ++p)
            acc[j][p] = floatx4_t{0.0f, 0.0f, 0.0f, 0.0f};
    u32x4_t wv[TN][4], xv[NP][4];
    auto load_w = [&](int q) {
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii)
                wv[j][ii] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(W + woff[j][ii] + (q << 7)));
    };
    auto load_x = [&](int q) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                xv[p][i] = *reinterpret_cast<const u32x4_t *>(X + ((((int64_t)q * X_PACKS_MAX + p) * 4 + i) << 9));
    };
    int q = ks0 + wave;
    if (q < ks1) {
        load_w(q);
        load_x(q);
    }
    for (; q < ks1; q += NW) {
        // this k-step's weights into the staging tile, then the next k-step's
        // weight loads go out.  Its activations (cache hits) are requested
        // only once this k-step's MFMAs have read theirs, so one set of
        // activation registers serves both: at three packings that keeps the
        // four-tile kernel at two waves per SIMD.
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int ii = 0; ii < 4; ++ii) {
                const int row = 4 * ii + lrow;
                *reinterpret_cast<u32x4_t *>(wl + j * 2048 + row * 128 + ((lch ^ row) << 3)) = wv[j][ii];
            }
        if (q + NW < ks1)
            load_w(q + NW);
        // the staging tile is private to this wave, whose LDS accesses run in
        // program order; the fences only keep the compiler from reordering them
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ch = (4 * i + kg) ^ r16;
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const u32x4_t w = *reinterpret_cast<const u32x4_t *>(wl + j * 2048 + r16 * 128 + (ch << 3));
#pragma unroll
                for (int p = 0; p < NP; ++p)
                    acc[j][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, w),
                                                                        __builtin_bit_cast(bf16x8_t, xv[p][i]),
                                                                        acc[j][p], 0, 0, 0);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        __builtin_amdgcn_sched_barrier(0);
        if (q + NW < ks1)
            load_x(q + NW);
    }

    // D[n_local][c]: lane l holds rows 4 (l / 16) + v, column l % 16.  The
    // reduction reuses the staging memory once every wave is done with it.
    __syncthreads();
    float *red = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                red[(wave * TN * 16 + 16 * j + 4 * kg + v) * RC + 16 * p + r16] = acc[j][p][v];
    __syncthreads();
    // fold the waves, then the terms (hi first): fin[n][m] = sum_t sum_w
    for (int o = tid; o < TN * 256; o += NW * 64) {
        const int ni = o >> 4, mi = o & 15;
        float v = 0.0f;
        if (mi < M) {
#pragma unroll
            for (int t = 0; t < X_TERMS; ++t) {
                const int c = t * M + mi;
                if (c < NP * 16)
#pragma unroll
                    for (int w = 0; w < NW; ++w)
                        v += red[(w * TN * 16 + ni) * RC + c];
            }
        }
        fin[o] = v;
    }
    if (tid < 16) {
        // RMSNorm: the fragments hold g * h; the slices' sums of h^2, in order
        float v = 1.0f;
        if (a.ssq && tid < M) {
            float ss = 0.0f;
            for (int sl = 0; sl < a.ssq_slices; ++sl)
                ss += a.ssq[tid * a.ssq_slices + sl];
            v = 1.0f / sqrtf(ss / (float)a.K + a.eps);
        }
        inv_s[tid] = v;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int t = grp * TN + j;
        if (t < n_tiles)
            run_epilogue<uint16_t, EPI>(a, fin + 256 * j, 16, 16, inv_s, t, M);
    }
}

// ---------------------------------------------------------------------------
// Activations for the MFMA path, one work-group per (row, slice of
// PREP_SLICE elements): the pending split-K partials of the last output
// projection are added into h (in split order), u = g * h (or h without a
// gain) is split into X_TERMS bf16 terms in fragment layout, and the
// slice's sum of h^2 goes to ssq[row][slice].  The consuming kernel sums
// the slices in order and divides its outputs by rms(h) itself, so no
// work-group needs the whole row and every slice is one round trip.

template <typename TW>
__global__ __launch_bounds__(PREP_SLICE / 4) void k_prep_norm(float *h, int64_t ldh, const TW *g, int K,
                                                              const DevCtl *ctl, uint16_t *xs, const float *part,
                                                              int n_part, float *ssq) {
    __shared__ float red[PREP_SLICE / 256];
    const int r = blockIdx.x, sl = blockIdx.y, M = ctl->m;
    if (r >= M)
        return;
    const int tid = threadIdx.x, k4 = sl * (PREP_SLICE / 4) + tid;
    const bool ok = 4 * k4 < K;
    float4 *hr = reinterpret_cast<float4 *>(h + (int64_t)r * ldh);
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (ok) {
        v = hr[k4];
        if (n_part > 0) {
            // every load of the element is issued before the adds
            float4 p[8];
#pragma unroll
            for (int sp = 0; sp < 8; ++sp)
                if (sp < n_part)
                    p[sp] = reinterpret_cast<const float4 *>(part + ((int64_t)sp * MAX_ROWS + r) * K)[k4];
#pragma unroll
            for (int sp = 0; sp < 8; ++sp)
                if (sp < n_part) {
                    v.x += p[sp].x;
                    v.y += p[sp].y;
                    v.z += p[sp].z;
                    v.w += p[sp].w;
                }
            hr[k4] = v;
        }
    }
    if (g) {
        float ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, v.w * v.w)));
        ss = wave_sum(ss);
        if ((tid & 63) == 0)
            red[tid >> 6] = ss;
        __syncthreads();
        if (tid == 0) {
            float t = 0.0f;
            for (int w = 0; w < PREP_SLICE / 256; ++w)
                t += red[w];
            ssq[r * gridDim.y + sl] = t;
        }
    }
    if (!ok)
        return;
    float u[4] = {v.x, v.y, v.z, v.w};
    uint16_t t[X_TERMS][4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (g) {
            float gk;
            if constexpr (sizeof(TW) == 2)
                gk = bf2f(g[4 * k4 + e]);
            else
                gk = g[4 * k4 + e];
            u[e] *= gk;
        }
        const uint16_t hi = bf16_rne_bits(u[e]);
        const float r1 = u[e] - bf2f(hi);
        const uint16_t mid = bf16_rne_bits(r1);
        t[0][e] = hi;
        t[1][e] = mid;
        t[2][e] = bf16_rne_bits(r1 - bf2f(mid));
    }
    // four consecutive k stay contiguous in the fragment layout
#pragma unroll
    for (int i = 0; i < X_TERMS; ++i) {
        uint2 pk;
        pk.x = t[i][0] | ((uint32_t)t[i][1] << 16);
        pk.y = t[i][2] | ((uint32_t)t[i][3] << 16);
        *reinterpret_cast<uint2 *>(xs + xfrag_off(i, r, 4 * k4, M)) = pk;
    }
}

hipError_t launch_prep_norm(float *h, int64_t ldh, const void *gain, bool bf16, int K, const DevCtl *ctl,
                            uint16_t *xs, const float *part, int n_part, float *ssq, hipStream_t s) {
    if ((K & 127) || (ldh & 3) || n_part > 8 || (gain && !ssq))
        return hipErrorInvalidValue;
    const dim3 grid(MAX_ROWS, prep_slices(K)), block(PREP_SLICE / 4);
    if (bf16)
        hipLaunchKernelGGL(k_prep_norm<uint16_t>, grid, block, 0, s, h, ldh, reinterpret_cast<const uint16_t *>(gain),
                           K, ctl, xs, part, n_part, ssq);
    else
        hipLaunchKernelGGL(k_prep_norm<float>, grid, block, 0, s, h, ldh, reinterpret_cast<const float *>(gain), K,
                           ctl, xs, part, n_part, ssq);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// dispatch

// A launch, with the optional start/stop events attached to the dispatch
// itself: they take the kernel's own start and end times and add no packets
// to the stream.
static void launch_k(void (*kern)(LinearArgs), dim3 grid, dim3 block, hipStream_t s, const LaunchTiming &t,
                     const LinearArgs &a) {
    if (t.start)
        hipExtLaunchKernelGGL(kern, grid, block, 0, s, t.start, t.stop, 0, a);
    else
        hipLaunchKernelGGL(kern, grid, block, 0, s, a);
}

template <typename TW, int MR, int R, int NT = 256, int U = 1>
static hipError_t launch_valu(const LinearArgs &a, int epi, int n_tiles, hipStream_t s, const LaunchTiming &t) {
    dim3 grid(n_tiles), block(NT);
    const bool norm = a.gain != nullptr;
    switch (epi) {
    case EPI_STORE:
        if (norm)
            launch_k(k_linear_valu<TW, MR, R, EPI_STORE, true, NT, U>, grid, block, s, t, a);
        else
            launch_k(k_linear_valu<TW, MR, R, EPI_STORE, false, NT, U>, grid, block, s, t, a);
        break;
    case EPI_RESID:
        launch_k(k_linear_valu<TW, MR, R, EPI_RESID, false, NT, U>, grid, block, s, t, a);
        break;
    case EPI_SWIGLU:
        launch_k(k_linear_valu<TW, MR, R, EPI_SWIGLU, true, NT, U>, grid, block, s, t, a);
        break;
    case EPI_QKV:
        launch_k(k_linear_valu<TW, MR, R, EPI_QKV, true, NT, U>, grid, block, s, t, a);
        break;
    case EPI_HEAD:
        launch_k(k_linear_valu<TW, MR, R, EPI_HEAD, true, NT, U>, grid, block, s, t, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename TW, int MR>
static hipError_t launch_valu_r(const LinearArgs &a, int epi, int R, int n_tiles, hipStream_t s,
                                const LaunchTiming &t) {
    switch (R) {
    case 4:
        return launch_valu<TW, MR, 4>(a, epi, n_tiles, s, t);
    case 8:
        return launch_valu<TW, MR, 8>(a, epi, n_tiles, s, t);
    case 16:
        if constexpr (MR <= 4)
            return launch_valu<TW, MR, 16>(a, epi, n_tiles, s, t);
        return hipErrorInvalidValue;
    default:
        return hipErrorInvalidValue;
    }
}

// Two rows on one-wave tiles (bf16 weights): 4 weight rows with one or two
// chunks' loads in flight, or 8 rows with one (the plan picks per shape).
static hipError_t launch_valu_wave2(const LinearArgs &a, int epi, int R, int U, int n_tiles, hipStream_t s,
                                    const LaunchTiming &t) {
    if (R == 4 && U == 2)
        return launch_valu<uint16_t, 2, 4, 64, 2>(a, epi, n_tiles, s, t);
    if (R == 4 && U == 1)
        return launch_valu<uint16_t, 2, 4, 64, 1>(a, epi, n_tiles, s, t);
    if (R == 8 && U == 1)
        return launch_valu<uint16_t, 2, 8, 64, 1>(a, epi, n_tiles, s, t);
    return hipErrorInvalidValue;
}

template <int TN, int NW, int NP>
static hipError_t launch_mfma(const LinearArgs &a, int epi, int n_tiles, hipStream_t s, const LaunchTiming &t) {
    const int groups = (n_tiles + TN - 1) / TN;
    dim3 grid(groups * (epi == EPI_PARTIAL ? a.splits : 1)), block(NW * 64);
    switch (epi) {
    case EPI_PARTIAL:
        if (a.splits < 1 || !a.part)
            return hipErrorInvalidValue;
        launch_k(k_linear_mfma<EPI_PARTIAL, TN, NW, NP>, grid, block, s, t, a);
        break;
    case EPI_STORE:
        launch_k(k_linear_mfma<EPI_STORE, TN, NW, NP>, grid, block, s, t, a);
        break;
    case EPI_RESID:
        launch_k(k_linear_mfma<EPI_RESID, TN, NW, NP>, grid, block, s, t, a);
        break;
    case EPI_SWIGLU:
        launch_k(k_linear_mfma<EPI_SWIGLU, TN, NW, NP>, grid, block, s, t, a);
        break;
    case EPI_QKV:
        launch_k(k_linear_mfma<EPI_QKV, TN, NW, NP>, grid, block, s, t, a);
        break;
    case EPI_HEAD:
        launch_k(k_linear_mfma<EPI_HEAD, TN, NW, NP>, grid, block, s, t, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// The work-group shape follows the output kind and the packing count
// (mfma_shape_tn / mfma_shape_nw).
constexpr int MFMA_WIDE_TILES = 1600;

static hipError_t launch_mfma_np(const LinearArgs &a, int epi, int n_tiles, hipStream_t s,
                                 const LaunchTiming &t) {
    const int np = mfma_packs(a.max_rows);
    if (epi == EPI_PARTIAL) {
        switch (np) {
        case 1:
            return launch_mfma<mfma_shape_tn(EPI_PARTIAL, 1), mfma_shape_nw(EPI_PARTIAL, 1), 1>(a, epi, n_tiles, s, t);
        case 2:
            return launch_mfma<mfma_shape_tn(EPI_PARTIAL, 2), mfma_shape_nw(EPI_PARTIAL, 2), 2>(a, epi, n_tiles, s, t);
        case 3:
            return launch_mfma<mfma_shape_tn(EPI_PARTIAL, 3), mfma_shape_nw(EPI_PARTIAL, 3), 3>(a, epi, n_tiles, s, t);
        default:
            return hipErrorInvalidValue;
        }
    }
    switch (np) {
    case 1:
        return launch_mfma<mfma_shape_tn(EPI_STORE, 1), mfma_shape_nw(EPI_STORE, 1), 1>(a, epi, n_tiles, s, t);
    case 2:
        return launch_mfma<mfma_shape_tn(EPI_STORE, 2), mfma_shape_nw(EPI_STORE, 2), 2>(a, epi, n_tiles, s, t);
    case 3:
        // Three packings on a wide gate/up or lm-head: eight tiles per
        // work-group halve the activation-fragment loads per weight byte.
        // Measured at the 13B shapes, 13 rows: gate/up (1728 tiles) 57.9 ->
        // 53.2 us, lm-head (2000 tiles) 60.7 -> 58.0; QKV (960 tiles, 120
        // work-groups of eight) 33.0 -> 50.6, and at 4 or 8 rows eight tiles
        // lose everywhere.
        if ((epi == EPI_SWIGLU || epi == EPI_HEAD) && n_tiles >= MFMA_WIDE_TILES)
            return launch_mfma<8, 4, 3>(a, epi, n_tiles, s, t);
        return launch_mfma<mfma_shape_tn(EPI_STORE, 3), mfma_shape_nw(EPI_STORE, 3), 3>(a, epi, n_tiles, s, t);
    default:
        return hipErrorInvalidValue;
    }
}

hipError_t launch_head_finalize(const LinearArgs &a, int n_tiles, hipStream_t s) {
    LinearArgs b = a;
    b.n_tiles = n_tiles;
    hipLaunchKernelGGL(k_head_finalize, dim3(1), dim3(HF_THREADS), 0, s, b);
    return hipGetLastError();
}

hipError_t launch_linear(const LinearArgs &a, int epi, bool bf16, int path, int rows_per_tile, int n_tiles,
                         hipStream_t s, const LaunchTiming &t, int chunks) {
    if (n_tiles <= 0)
        return hipSuccess;
    if (path == PATH_MFMA) {
        // n_tiles counts 16-row tiles; the work-group shape is chosen here
        (void)rows_per_tile;
        if (!bf16 || (a.K & 127))
            return hipErrorInvalidValue;
        if (!a.Xs || a.max_rows < 1 || a.max_rows > MAX_ROWS)
            return hipErrorInvalidValue;
        if ((int64_t)a.N * a.K >= ((int64_t)1 << 32))  // 32-bit weight offsets
            return hipErrorInvalidValue;
        LinearArgs b = a;
        b.n_tiles = n_tiles;
        return launch_mfma_np(b, epi, n_tiles, s, t);
    }
    if (path == PATH_GEMV_FP8) {
        if (!bf16 || (a.K & 15) || !a.wexp)
            return hipErrorInvalidValue;
        if (rows_per_tile == 4)
            return launch_fp8_r<4>(a, epi, n_tiles, s, t);
        if (rows_per_tile == 8)
            return launch_fp8_r<8>(a, epi, n_tiles, s, t);
        return hipErrorInvalidValue;
    }
    if (a.K & 7)
        return hipErrorInvalidValue;
    if (path == PATH_GEMV)
        return bf16 ? launch_valu_r<uint16_t, 1>(a, epi, rows_per_tile, n_tiles, s, t)
                    : launch_valu_r<float, 1>(a, epi, rows_per_tile, n_tiles, s, t);
    if (path == PATH_VALU2)
        return bf16 ? launch_valu_r<uint16_t, 2>(a, epi, rows_per_tile, n_tiles, s, t)
                    : launch_valu_r<float, 2>(a, epi, rows_per_tile, n_tiles, s, t);
    if (path == PATH_WAVE2)
        return bf16 ? launch_valu_wave2(a, epi, rows_per_tile, chunks ? chunks : wave2_default_chunks(rows_per_tile),
                                        n_tiles, s, t)
                    : hipErrorInvalidValue;
    return bf16 ? launch_valu_r<uint16_t, 16>(a, epi, rows_per_tile, n_tiles, s, t)
                : launch_valu_r<float, 16>(a, epi, rows_per_tile, n_tiles, s, t);
}

}  // namespace sdk
