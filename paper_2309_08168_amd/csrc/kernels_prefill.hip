// Large-M forward: the prompt prefill that fills the KV cache before the
// first draft (Algorithm 2 starts from a cache holding the prompt), and
// long forwards in general.  With hundreds of rows the linear layers are
// dense contractions, 2 M N K flops per N K weight bytes, so they run on
// matrix cores:
//   - k_pf_gemm: C = A W^T with the float32 activations split into X_TERMS
//     bfloat16 terms (exact for float32 values), 256 x 128 output tiles,
//     stages of 32 k staged through double-buffered LDS in MFMA fragment
//     order, v_mfma 16x16x32 bf16; tiles are ordered so the work-groups one
//     XCD runs together share their weight and activation slices in that
//     XCD's L2; narrow residual updates split the reduction into partials;
//   - k_pf_gemm_wide: the same product on 256 x 256 (or 256 x 224) tiles
//     with the operands loaded straight into LDS, for the layers with
//     enough tiles to fill the CUs, and for split residual updates that do;
//   - k_pf_attn: causal attention, one wave per 16 query rows of a head,
//     scores and the weighted sum of values on matrix cores with an online
//     softmax over 32-key blocks, the longest row blocks dispatched first and
//     spread evenly over the XCDs;
//   - small row kernels between them: embedding, RMSNorm + split (adding a
//     split residual update's partials first), rotary embedding + KV
//     append, SwiGLU + split.
#include "sd_internal.h"

#include <algorithm>

namespace sdk {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

__device__ __forceinline__ f32x4_t mfma16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

__device__ __forceinline__ float bf_to_f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// Terms of eight consecutive values, each packed as 8 bf16 (one 16-byte word).
__device__ __forceinline__ void split8(const float (&x)[8], u32x4_t (&t)[X_TERMS]) {
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
#pragma unroll
        for (int j = 0; j < 4; ++j)
            t[i][j] = (uint32_t)h[i][2 * j] | ((uint32_t)h[i][2 * j + 1] << 16);
}

// ---------------------------------------------------------------------------
// GEMM
//
// Work-group tile: 256 weight rows (output columns) x 128 activation rows,
// 8 waves (2 per SIMD, so one wave's MFMAs run while the other waits).
// Each 32-k stage is staged through LDS in fragment order: every 16 x 32
// MFMA operand block is 1 KB with lane l's 16 bytes at offset 16 l, so a
// fragment read is one contiguous 1 KB read and the staging writes of each
// 8-lane group are 128 contiguous bytes (bank-conflict free both ways).
// The weight tile is read once per 128 rows; each activation term block
// once per 256 columns.

constexpr int GB_N = 256;  // weight rows (output columns) per work-group
constexpr int GB_M = 128;  // activation rows per work-group
constexpr int GB_K = 32;   // k per stage: one MFMA k-step
constexpr int G_THREADS = 512;

// Offset (bf16 elements) of the 16-byte chunk kc of row r in a stage buffer.
__device__ __forceinline__ int frag_off(int r, int kc) { return (r >> 4) * 512 + ((r & 15) + 16 * kc) * 8; }

// NWN x NWM waves (NWN along the weight rows); DEPTH stages of operands in
// flight in registers; EPI_PARTIAL writes the split's partial tile to
// part[blockIdx split][m][n].
template <int EPI, int NWN, int NWM, int DEPTH>
__global__ __launch_bounds__(G_THREADS, 2) void k_pf_gemm(PfGemmArgs a) {
    constexpr int T = X_TERMS;
    constexpr int WN = GB_N / NWN, WM = GB_M / NWM;  // a wave's share
    constexpr int NT = WN / 16, MT = WM / 16;        // 16 x 16 output tiles per wave
    constexpr int W_PT = GB_N * 4 / G_THREADS;       // staging chunks per thread: weights
    constexpr int A_PT = T * GB_M * 4 / G_THREADS;   // staging chunks per thread: activation terms
    static_assert(NWN * NWM * 64 == G_THREADS && W_PT * G_THREADS == GB_N * 4 && A_PT * G_THREADS == T * GB_M * 4,
                  "tile split");
    static_assert(DEPTH == 1 || DEPTH == 2, "stages in flight");
    __shared__ __attribute__((aligned(16))) uint16_t ws[2][GB_N * GB_K];
    __shared__ __attribute__((aligned(16))) uint16_t as[2][T * GB_M * GB_K];

    const int M = a.M, N = a.N, K = a.K;
    // Tile and k-split of this work-group.  Work-groups are dealt to the 8
    // XCDs in turn, so each XCD gets a contiguous range of tile indices, and
    // the range is walked in groups of 4 row tiles: the tiles one XCD runs
    // at a time form a compact block whose operand slices its L2 holds.
    const int TM = (M + GB_M - 1) / GB_M, TN = (N + GB_N - 1) / GB_N, TT = TM * TN * a.splits;
    const int per = (TT + 7) / 8;
    int L = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (L >= TT)
        return;  // uniform over the work-group
    const int split = L % a.splits;
    L /= a.splits;
    const int GM = TM < 4 ? TM : 4;
    const int grp_i = L / (GM * TN), first = grp_i * GM, gm = min(TM - first, GM);
    const int in = L - grp_i * GM * TN;
    const int m0 = (first + in % gm) * GB_M, n0 = (in / gm) * GB_N;
    const int S_all = (K + GB_K - 1) / GB_K, S_per = (S_all + a.splits - 1) / a.splits;
    const int s_begin = split * S_per, S = max(0, min(S_all - s_begin, S_per));

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int wn = wave % NWN, wm = wave / NWN;

    // staging chunk c: row 8 (c / 32) + c % 8, k chunk (c / 8) % 4.  Every
    // load is unconditional (clamped rows, clamped k, stages past the end
    // reload the last one); chunks past K become zeros on the way into LDS.
    u32x4_t wr[DEPTH][W_PT], ar[DEPTH][A_PT];
    auto gload = [&](u32x4_t(&w)[W_PT], u32x4_t(&x)[A_PT], int stage) {
        const int k0 = (s_begin + min(stage, max(S - 1, 0))) * GB_K;
#pragma unroll
        for (int i = 0; i < W_PT; ++i) {
            const int c = tid + G_THREADS * i, row = 8 * (c >> 5) + (c & 7), k = k0 + 8 * ((c >> 3) & 3);
            w[i] = *reinterpret_cast<const u32x4_t *>(a.W + (int64_t)min(n0 + row, N - 1) * K + min(k, K - 8));
        }
#pragma unroll
        for (int i = 0; i < A_PT; ++i) {
            const int c = tid + G_THREADS * i, t = c / (GB_M * 4), rem = c - t * GB_M * 4;
            const int row = 8 * (rem >> 5) + (rem & 7), k = k0 + 8 * ((rem >> 3) & 3);
            x[i] = *reinterpret_cast<const u32x4_t *>(a.A + t * a.a_term + (int64_t)min(m0 + row, M - 1) * a.lda +
                                                      min(k, K - 8));
        }
    };
    auto lstore = [&](int buf, const u32x4_t(&w)[W_PT], const u32x4_t(&x)[A_PT], int stage) {
        const int k0 = (s_begin + stage) * GB_K;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < W_PT; ++i) {
            const int c = tid + G_THREADS * i, row = 8 * (c >> 5) + (c & 7), kc = (c >> 3) & 3;
            *reinterpret_cast<u32x4_t *>(&ws[buf][frag_off(row, kc)]) = k0 + 8 * kc < K ? w[i] : zero;
        }
#pragma unroll
        for (int i = 0; i < A_PT; ++i) {
            const int c = tid + G_THREADS * i, t = c / (GB_M * 4), rem = c - t * GB_M * 4;
            const int row = 8 * (rem >> 5) + (rem & 7), kc = (rem >> 3) & 3;
            *reinterpret_cast<u32x4_t *>(&as[buf][frag_off(t * GB_M + row, kc)]) = k0 + 8 * kc < K ? x[i] : zero;
        }
    };

    f32x4_t acc[NT][MT];
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j)
            acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    auto compute = [&](int buf) {
        u32x4_t wf[NT], af[MT][T];
#pragma unroll
        for (int i = 0; i < NT; ++i)
            wf[i] = *reinterpret_cast<const u32x4_t *>(&ws[buf][(wn * NT + i) * 512 + lane * 8]);
#pragma unroll
        for (int j = 0; j < MT; ++j)
#pragma unroll
            for (int t = 0; t < T; ++t)
                af[j][t] =
                    *reinterpret_cast<const u32x4_t *>(&as[buf][(t * (GB_M / 16) + wm * MT + j) * 512 + lane * 8]);
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int i = 0; i < NT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j)
                    acc[i][j] = mfma16(wf[i], af[j][t], acc[i][j]);
    };

    // step s: issue the loads of stage s + DEPTH into the set stage s came
    // from, multiply stage s (LDS buffer s % 2), move stage s + 1 from its
    // register set into the other buffer, barrier
    if (S > 0) {
        gload(wr[0], ar[0], 0);
        if constexpr (DEPTH == 2)
            gload(wr[DEPTH - 1], ar[DEPTH - 1], 1);
        lstore(0, wr[0], ar[0], 0);
    }
    __syncthreads();
    if constexpr (DEPTH == 1) {
        for (int s = 0; s < S; ++s) {
            gload(wr[0], ar[0], s + 1);
            compute(s & 1);
            if (s + 1 < S)
                lstore((s & 1) ^ 1, wr[0], ar[0], s + 1);
            __syncthreads();
        }
    } else {
        for (int s = 0; s < S; s += 2) {
            gload(wr[0], ar[0], s + 2);
            compute(0);
            if (s + 1 < S)
                lstore(1, wr[DEPTH - 1], ar[DEPTH - 1], s + 1);
            __syncthreads();
            if (s + 1 >= S)
                break;
            gload(wr[DEPTH - 1], ar[DEPTH - 1], s + 3);
            compute(1);
            if (s + 2 < S)
                lstore(0, wr[0], ar[0], s + 2);
            __syncthreads();
        }
    }

    // lane holds C^T[n0 + wn WN + 16 i + 4 grp + v][m0 + wm WM + 16 j + col]
    const int col = lane & 15, grp = lane >> 4;
    float *C = EPI == EPI_PARTIAL ? a.part + (int64_t)split * M * a.ldc : a.C;
    const bool vec = (a.ldc & 3) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
#pragma unroll
    for (int i = 0; i < NT; ++i) {
        const int n = n0 + wn * WN + 16 * i + 4 * grp;
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int m = m0 + wm * WM + 16 * j + col;
            if (m >= M || n >= N)
                continue;
            float *c = C + (int64_t)m * a.ldc + n;
            if (vec && n + 3 < N) {
                f32x4_t v = acc[i][j];
                if constexpr (EPI == EPI_RESID)
                    v += *reinterpret_cast<const f32x4_t *>(c);
                *reinterpret_cast<f32x4_t *>(c) = v;
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (n + v < N)
                        c[v] = EPI == EPI_RESID ? c[v] + acc[i][j][v] : acc[i][j][v];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Wide GEMM with direct-to-LDS operand loads
//
// The same product and accumulation order as k_pf_gemm (bit-identical
// results; plain stores) for layers with at least 128 tiles of 256 x 256:
// 256 activation rows x 256 (or 224) weight rows per work-group as 16 waves
// (four per SIMD; eight waves of 128 x 64 were 1-4% slower), 32-k stages.
// Operands go from global memory straight into LDS with
// global_load_lds_dwordx4: one instruction fills one 1 KB fragment block
// (lane l's 16 bytes at 16 l), so no registers stage them and no second
// pass writes LDS.  Two 64 KB stage buffers: the loads of stage s + 1 are
// issued right after the barrier that ends stage s - 1.  The barrier is a
// bare s_barrier: a release fence before it would also wait for the next
// stage's loads.  K must be a multiple of 32.

constexpr int GW_M = 256;                                        // activation rows per work-group
constexpr int GW_WAVES = 16;                                     // waves per work-group
constexpr int GW_THREADS = 64 * GW_WAVES;
constexpr int GW_MIN_TILES = 128;                                // tiles that make a launch "wide"
constexpr int GW_MIN_SPLIT_GROUPS = 160;                         // work-groups of a wide split reduction
constexpr int GW_BLOCKS = GB_N / 16 + X_TERMS * GW_M / 16;       // 1 KB fragment blocks per stage (at most)
constexpr int GW_PER = GW_BLOCKS / GW_WAVES;                     // load instructions per wave per stage
static_assert(GW_BLOCKS % GW_WAVES == 0, "blocks per wave");

// s_waitcnt immediate (gfx9 layout: vmcnt bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8) that waits for vmcnt 0 and leaves the other counters alone
constexpr int WAIT_VMCNT0 = (7 << 4) | (15 << 8);

__device__ __forceinline__ void load_to_lds16(const uint16_t *g, uint16_t *l) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)g,
                                     (__attribute__((address_space(3))) void *)l, 16, 0, 0);
}

// BN: weight rows per tile, 256 (4 x 4 waves of 64 x 64) or 224 (2 x 8
// waves of 112 x 32, 14 weight blocks per stage, the last two load slots of
// a stage idle).  EPI_SWIGLU (W = [gate; up], N = 2 F): a tile takes the
// gate and the up rows of the same BN / 2 columns f of the MLP, the waves
// holding up pass their sums to the waves holding gate through LDS, and
// those write silu(gate) * up as terms.
template <int EPI, int BN>
__global__ __launch_bounds__(GW_THREADS, 4) void k_pf_gemm_wide(PfGemmArgs a) {
    static_assert(BN == 256 || BN == 224, "tile width");
    constexpr int T = X_TERMS, NWN = BN == 256 ? 4 : 2, NWM = GW_WAVES / NWN;
    constexpr int WN = BN / NWN, WM = GW_M / NWM;
    constexpr int NT = WN / 16, MT = WM / 16;
    constexpr int NBW = BN / 16;                       // weight blocks per stage
    constexpr int NB = NBW + X_TERMS * GW_M / 16;      // blocks per stage
    static_assert(NB <= GW_BLOCKS && NT * 16 == WN && MT * 16 == WM, "tile split");
    __shared__ __attribute__((aligned(1024))) uint16_t lds[2 * GW_BLOCKS * 512];

    constexpr bool SWI = EPI == EPI_SWIGLU;
    constexpr int BC = SWI ? BN / 2 : BN;              // output columns per tile
    const int M = a.M, N = a.N, K = a.K, F = N / 2;
    const int NC = SWI ? F : N;                        // output columns
    // tile and k-split order as in k_pf_gemm: each XCD a contiguous range,
    // walked in groups of up to 4 row tiles
    const int TM = (M + GW_M - 1) / GW_M, TN = (NC + BC - 1) / BC, TT = TM * TN * a.splits;
    const int per = (TT + 7) / 8;
    int L = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (L >= TT)
        return;  // uniform over the work-group
    const int split = L % a.splits;
    L /= a.splits;
    const int GM = TM < 4 ? TM : 4;
    const int grp_i = L / (GM * TN), first = grp_i * GM, gm = min(TM - first, GM);
    const int in = L - grp_i * GM * TN;
    const int m0 = (first + in % gm) * GW_M, n0 = (in / gm) * BC;  // SWI: n0 is the first f
    // the split's stages (possibly none: its partial tile is then zeros)
    const int S_all = K / GB_K, S_per = (S_all + a.splits - 1) / a.splits;
    const int s_begin = split * S_per, S = max(0, min(S_all - s_begin, S_per));

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int wn = wave % NWN, wm = wave / NWN;

    // block b of a stage: b < NBW the weight rows n0 + 16 b .., else term t
    // of activation rows m0 + 16 rg ..; lane l loads row 16 b + l % 16,
    // k chunk l / 16 (rows past the end read the last row: never stored)
    const uint16_t *src[GW_PER];
#pragma unroll
    for (int i = 0; i < GW_PER; ++i) {
        const int b = min(wave + GW_WAVES * i, NB - 1);  // slots past NB load nothing (below)
        if (b < NBW) {
            int row;
            if constexpr (SWI)  // gate rows f, then up rows F + f
                row = (b < NBW / 2 ? 0 : F) + min(n0 + 16 * (b % (NBW / 2)) + (lane & 15), F - 1);
            else
                row = min(n0 + 16 * b + (lane & 15), N - 1);
            src[i] = a.W + (int64_t)row * K + 8 * (lane >> 4);
        } else {
            const int c = b - NBW, t = c / (GW_M / 16), rg = c % (GW_M / 16);
            src[i] = a.A + t * a.a_term + (int64_t)min(m0 + 16 * rg + (lane & 15), M - 1) * a.lda + 8 * (lane >> 4);
        }
    }
    auto issue = [&](int stage) {
        uint16_t *dst = lds + (stage & 1) * GW_BLOCKS * 512;
#pragma unroll
        for (int i = 0; i < GW_PER; ++i)
            if (NB % GW_WAVES == 0 || wave + GW_WAVES * i < NB)  // uniform over the wave
                load_to_lds16(src[i] + (s_begin + stage) * GB_K, dst + (wave + GW_WAVES * i) * 512);
    };

    f32x4_t acc[NT][MT];
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j)
            acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    if (S > 0)
        issue(0);
    for (int s = 0; s < S; ++s) {
        // this wave's stage-s blocks have landed (nothing else is in flight)
        __builtin_amdgcn_s_waitcnt(WAIT_VMCNT0);
        // all waves' blocks have landed and every wave's reads of the other
        // buffer (stage s - 1) have returned
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (s + 1 < S)
            issue(s + 1);
        const uint16_t *ws = lds + (s & 1) * GW_BLOCKS * 512, *as = ws + NBW * 512;
        u32x4_t wf[NT], af[MT][T];
#pragma unroll
        for (int i = 0; i < NT; ++i)
            wf[i] = *reinterpret_cast<const u32x4_t *>(&ws[(wn * NT + i) * 512 + lane * 8]);
#pragma unroll
        for (int j = 0; j < MT; ++j)
#pragma unroll
            for (int t = 0; t < T; ++t)
                af[j][t] = *reinterpret_cast<const u32x4_t *>(&as[(t * (GW_M / 16) + wm * MT + j) * 512 + lane * 8]);
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int i = 0; i < NT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j)
                    acc[i][j] = mfma16(wf[i], af[j][t], acc[i][j]);
    }

    // lane holds C^T[n0 + wn WN + 16 i + 4 grp + v][m0 + wm WM + 16 j + col]
    // (EPI_PARTIAL: of the split's partial sum, part[split][m][n])
    static_assert(EPI == EPI_STORE || EPI == EPI_PARTIAL || EPI == EPI_SWIGLU, "stores only");
    const int col = lane & 15, grp = lane >> 4;
    if constexpr (SWI) {
        // wave column wn < NWN / 2 holds gate, wn + NWN / 2 up of the same f
        constexpr int HALF = NWN / 2, SLOT = NT * MT * 64;  // f32x4 per up wave
        static_assert(NWM * HALF * SLOT * 16 <= (int)sizeof(lds), "exchange fits the stage buffers");
        f32x4_t *xl = reinterpret_cast<f32x4_t *>(lds);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // all reads of the stages done
        if (wn >= HALF) {
#pragma unroll
            for (int i = 0; i < NT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j)
                    xl[(wm * HALF + wn - HALF) * SLOT + (i * MT + j) * 64 + lane] = acc[i][j];
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (wn >= HALF)
            return;
        const bool vec = (F & 3) == 0 && (a.x_term & 3) == 0 && (reinterpret_cast<uintptr_t>(a.xout) & 7) == 0;
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const int f = n0 + wn * WN + 16 * i + 4 * grp;
#pragma unroll
            for (int j = 0; j < MT; ++j) {
                const int m = m0 + wm * WM + 16 * j + col;
                const f32x4_t up = xl[(wm * HALF + wn) * SLOT + (i * MT + j) * 64 + lane];
                if (m >= M || f >= F)
                    continue;
                uint16_t t4[T][4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float g = acc[i][j][v];
                    uint16_t t3[T];
                    split3(g / (1.0f + expf(-g)) * up[v], t3);
#pragma unroll
                    for (int q = 0; q < T; ++q)
                        t4[q][v] = t3[q];
                }
                uint16_t *o = a.xout + (int64_t)m * F + f;
                if (vec && f + 3 < F) {
#pragma unroll
                    for (int q = 0; q < T; ++q) {
                        const u32x2_t w = {(uint32_t)t4[q][0] | ((uint32_t)t4[q][1] << 16),
                                           (uint32_t)t4[q][2] | ((uint32_t)t4[q][3] << 16)};
                        *reinterpret_cast<u32x2_t *>(o + q * a.x_term) = w;
                    }
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (f + v < F)
#pragma unroll
                            for (int q = 0; q < T; ++q)
                                o[q * a.x_term + v] = t4[q][v];
                }
            }
        }
        return;
    }
    float *C = EPI == EPI_PARTIAL ? a.part + (int64_t)split * M * a.ldc : a.C;
    const bool vec = (a.ldc & 3) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
#pragma unroll
    for (int i = 0; i < NT; ++i) {
        const int n = n0 + wn * WN + 16 * i + 4 * grp;
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int m = m0 + wm * WM + 16 * j + col;
            if (m >= M || n >= N)
                continue;
            float *c = C + (int64_t)m * a.ldc + n;
            if (vec && n + 3 < N) {
                *reinterpret_cast<f32x4_t *>(c) = acc[i][j];
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    if (n + v < N)
                        c[v] = acc[i][j][v];
            }
        }
    }
}

// C[m][n] += part[0][m][n] + part[1][m][n] + ..., in split order.
__global__ __launch_bounds__(256) void k_pf_split_sum(const float *part, int splits, int64_t stride, float *C,
                                                      int64_t n_elems) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_elems; i += (int64_t)gridDim.x * 256) {
        float v = part[i];
        for (int s = 1; s < splits; ++s)
            v += part[(int64_t)s * stride + i];
        C[i] += v;
    }
}

// ---------------------------------------------------------------------------
// Causal attention.  Work-group (64-row block, head): wave w takes query rows
// r0 .. r0 + 15 and walks the keys [0, start + its last row] in blocks of
// 32.  Score tile t, row i holds key kb + 16 t + 4 (i % 4) + i / 4, so lane
// group G ends up with keys kb + 16 t + 4 v + G, which are exactly the
// reduction slots 8 G + 4 t + v that the lane supplies to the value MFMA:
// the probabilities never leave their lanes.  Values are staged in the
// wave's LDS tile (row pitch head_dim + 16, conflict-free) and gathered in
// that key order.

constexpr int PA_KB = 32;

template <int DH>
__global__ __launch_bounds__(256) void k_pf_attn(PfAttnArgs a) {
    constexpr int T = X_TERMS;
    constexpr int ES = DH / 32;     // 32-wide slices of head_dim (score MFMAs)
    constexpr int ET = DH / 16;     // 16-wide tiles of head_dim (value MFMAs)
    constexpr int VP = DH + 16;     // LDS pitch of a value row, bf16
    constexpr int LPR = DH / 8;     // lanes per value row (16-byte loads)
    constexpr int RPI = 64 / LPR;   // value rows per load instruction
    constexpr int NVJ = PA_KB / RPI;
    __shared__ __attribute__((aligned(16))) uint16_t vt[4][PA_KB * VP];

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 15, grp = lane >> 4;
    // Work-group i takes head i % H and row block TM - 1 - i / H: the
    // longest row blocks (most keys) start first, and consecutive indices,
    // which the dispatcher deals to the 8 XCDs in turn, carry the same mix of
    // row blocks on every XCD.  (With the row block as the fast grid index,
    // row blocks x and x + 8 of every head landed on one XCD: the one holding
    // the last row blocks had 2.4 times the work of the lightest.)
    const int TM = (a.M + 63) / 64;
    const int head = (int)(blockIdx.x % a.n_heads), g = head / (a.n_heads / a.n_kv_heads);
    const int r0 = (TM - 1 - (int)(blockIdx.x / a.n_heads)) * 64 + wave * 16;
    if (r0 >= a.M)
        return;  // uniform over the wave; the waves never synchronise
    const bool qok = r0 + col < a.M;
    const int rq = min(r0 + col, a.M - 1);
    const int qpos = a.start + rq;
    const int kend = a.start + min(r0 + 15, a.M - 1) + 1;  // keys some row of the wave sees
    const uint16_t *Kg = a.kcache + (int64_t)g * a.kv_head_stride;
    const uint16_t *Vg = a.vcache + (int64_t)g * a.kv_head_stride;
    uint16_t *vs = vt[wave];

    // query terms: B operand of the score MFMAs (dims x queries)
    u32x4_t qf[ES][T];
    {
        const float *qs = a.q + (int64_t)rq * a.ldq + (int64_t)head * DH + 8 * grp;
        const float scale = 1.0f / sqrtf((float)DH);
#pragma unroll
        for (int s = 0; s < ES; ++s) {
            const f32x4_t lo = reinterpret_cast<const f32x4_t *>(qs + 32 * s)[0];
            const f32x4_t hi = reinterpret_cast<const f32x4_t *>(qs + 32 * s)[1];
            float x[8];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                x[u] = lo[u] * scale;
                x[4 + u] = hi[u] * scale;
            }
            split8(x, qf[s]);
        }
    }

    float m_run = -INFINITY, l_run = 0.0f;
    f32x4_t oacc[ET];
#pragma unroll
    for (int et = 0; et < ET; ++et)
        oacc[et] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    for (int kb = 0; kb < kend; kb += PA_KB) {
        // keys past kend read the last key inside it: their scores are
        // masked and their weights are zero
        u32x4_t kf[2][ES], vr[NVJ];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int key = min(kb + 16 * t + 4 * (col & 3) + (col >> 2), kend - 1);
            const uint16_t *kp = Kg + (int64_t)key * DH + 8 * grp;
#pragma unroll
            for (int s = 0; s < ES; ++s)
                kf[t][s] = *reinterpret_cast<const u32x4_t *>(kp + 32 * s);
        }
#pragma unroll
        for (int j = 0; j < NVJ; ++j) {
            const int key = min(kb + j * RPI + lane / LPR, kend - 1);
            vr[j] = *reinterpret_cast<const u32x4_t *>(Vg + (int64_t)key * DH + 8 * (lane % LPR));
        }
        __builtin_amdgcn_sched_barrier(0);

        f32x4_t sacc[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            sacc[t] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int s = 0; s < ES; ++s)
#pragma unroll
                for (int i = 0; i < T; ++i)
                    sacc[t] = mfma16(kf[t][s], qf[s][i], sacc[t]);
        }
        // online softmax; slot u = 4 t + v of this lane is key kb + 16 t + 4 v + grp
        float sv[8], bm = -INFINITY;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int key = kb + 16 * (u >> 2) + 4 * (u & 3) + grp;
            sv[u] = key <= qpos ? sacc[u >> 2][u & 3] : -INFINITY;
            bm = fmaxf(bm, sv[u]);
        }
        bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
        bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
        const float m_new = fmaxf(m_run, bm);  // finite: key 0 is in the first block
        const float sc = expf(m_run - m_new);
        float p[8], ls = 0.0f;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            p[u] = expf(sv[u] - m_new);
            ls += p[u];
        }
        ls += __shfl_xor(ls, 16, 64);
        ls += __shfl_xor(ls, 32, 64);
        l_run = l_run * sc + ls;
        m_run = m_new;
        u32x4_t pf[T];
        split8(p, pf);

        // values of the block into the wave's tile (after the previous
        // block's reads), then O^T += V^T P^T tile by tile
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int j = 0; j < NVJ; ++j)
            *reinterpret_cast<u32x4_t *>(vs + (j * RPI + lane / LPR) * VP + 8 * (lane % LPR)) = vr[j];
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int et = 0; et < ET; ++et) {
            // A operand V^T: lane (col, grp) needs column 16 et + col of keys
            // kb + 16 (u >> 2) + 4 (u & 3) + grp, u = 0..7 (the score slots).
            // ds_read_b64_tr_b16 hands lane l of each 16-lane group element
            // l % 4 of the 8 bytes that lanes l / 4 + 4 k (k = 0..3) point at,
            // so lane r points at key kb + 16 I + 4 (r >> 2) + grp, columns
            // 16 et + 4 (r & 3) ..: two reads give the eight keys in order.
            uint32_t w[4];
#pragma unroll
            for (int I = 0; I < 2; ++I) {
                const uint16_t *src = vs + (16 * I + 4 * (col >> 2) + grp) * VP + 16 * et + 4 * (col & 3);
                const s16x4_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)src);
                w[2 * I] = (uint32_t)(uint16_t)r[0] | ((uint32_t)(uint16_t)r[1] << 16);
                w[2 * I + 1] = (uint32_t)(uint16_t)r[2] | ((uint32_t)(uint16_t)r[3] << 16);
            }
            const u32x4_t vf = {w[0], w[1], w[2], w[3]};
            oacc[et] *= sc;
#pragma unroll
            for (int i = 0; i < T; ++i)
                oacc[et] = mfma16(vf, pf[i], oacc[et]);
        }
    }

    // lane holds O^T[16 et + 4 grp + v][query col]; the terms of 4
    // consecutive elements go out as one 8-byte store per term
    if (qok) {
        const float inv = 1.0f / l_run;
#pragma unroll
        for (int et = 0; et < ET; ++et) {
            uint16_t t4[T][4];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                uint16_t s[T];
                split3(oacc[et][v] * inv, s);
#pragma unroll
                for (int i = 0; i < T; ++i)
                    t4[i][v] = s[i];
            }
            const int64_t e = (int64_t)rq * a.ldo + (int64_t)head * DH + 16 * et + 4 * grp;
#pragma unroll
            for (int i = 0; i < T; ++i) {
                const u32x2_t w = {(uint32_t)t4[i][0] | ((uint32_t)t4[i][1] << 16),
                                   (uint32_t)t4[i][2] | ((uint32_t)t4[i][3] << 16)};
                *reinterpret_cast<u32x2_t *>(a.out + i * a.out_term + e) = w;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Row kernels (one work-group per row)

__global__ __launch_bounds__(256) void k_pf_embed(const uint16_t *E, int d, const int32_t *tokens, float *h) {
    const int m = blockIdx.x;
    const uint16_t *e = E + (int64_t)tokens[m] * d;
    float *o = h + (int64_t)m * d;
    for (int k = threadIdx.x; k < d; k += 256)
        o[k] = bf_to_f(e[k]);
}

__global__ __launch_bounds__(256) void k_pf_norm_split(const float *h, int K, const uint16_t *gain, float eps,
                                                       uint16_t *out, int64_t out_term) {
    __shared__ float red[4];
    const int m = blockIdx.x, tid = threadIdx.x;
    const float *x = h + (int64_t)m * K;
    float ss = 0.0f;
    for (int k = 4 * tid; k < K; k += 4 * 256) {
        const f32x4_t v = *reinterpret_cast<const f32x4_t *>(x + k);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            ss = fmaf(v[j], v[j], ss);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        ss += __shfl_xor(ss, o, 64);
    if ((tid & 63) == 0)
        red[tid >> 6] = ss;
    __syncthreads();
    const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + eps);
    for (int k = 8 * tid; k < K; k += 8 * 256) {
        float u[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            u[j] = bf_to_f(gain[k + j]) * (x[k + j] * inv);
        u32x4_t t[X_TERMS];
        split8(u, t);
#pragma unroll
        for (int i = 0; i < X_TERMS; ++i)
            *reinterpret_cast<u32x4_t *>(out + i * out_term + (int64_t)m * K + k) = t[i];
    }
}

// h[m] += the split partials (in split order), then g * h / rms(h) as terms:
// the sums of k_pf_split_sum and the norm of k_pf_norm_split in one kernel
// (the second pass re-reads elements the work-group wrote before the
// barrier).
__global__ __launch_bounds__(256) void k_pf_fold_norm_split(float *h, const float *part, int splits, int64_t stride,
                                                            int K, const uint16_t *gain, float eps, uint16_t *out,
                                                            int64_t out_term) {
    __shared__ float red[4];
    const int m = blockIdx.x, tid = threadIdx.x;
    float *x = h + (int64_t)m * K;
    const float *p = part + (int64_t)m * K;
    float ss = 0.0f;
    // 16-byte loads (K is a multiple of 8): with 4-byte loads this pass over
    // the row and three partial planes took 40 us per 13B call
    for (int k = 4 * tid; k < K; k += 4 * 256) {
        f32x4_t v = *reinterpret_cast<const f32x4_t *>(p + k);
        for (int s = 1; s < splits; ++s)
            v += *reinterpret_cast<const f32x4_t *>(p + (int64_t)s * stride + k);
        const f32x4_t hn = *reinterpret_cast<const f32x4_t *>(x + k) + v;
        *reinterpret_cast<f32x4_t *>(x + k) = hn;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            ss = fmaf(hn[j], hn[j], ss);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        ss += __shfl_xor(ss, o, 64);
    if ((tid & 63) == 0)
        red[tid >> 6] = ss;
    __syncthreads();
    const float inv = 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + eps);
    for (int k = 8 * tid; k < K; k += 8 * 256) {
        float u[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            u[j] = bf_to_f(gain[k + j]) * (x[k + j] * inv);
        u32x4_t t[X_TERMS];
        split8(u, t);
#pragma unroll
        for (int i = 0; i < X_TERMS; ++i)
            *reinterpret_cast<u32x4_t *>(out + i * out_term + (int64_t)m * K + k) = t[i];
    }
}

__global__ __launch_bounds__(256) void k_pf_rope_kv(const float *qkv, int start, const float2 *rope, int H, int KVH,
                                                    int dh, float *q, uint16_t *kc, uint16_t *vc, int64_t stride) {
    const int m = blockIdx.x, pos = start + m, half = dh >> 1;
    const int nq = (H + 2 * KVH) * dh;
    const float *x = qkv + (int64_t)m * nq;
    // four pair indices i .. i + 3 of one head per step (half is a multiple
    // of 4): 16-byte loads and stores, 8-byte stores into the cache
    for (int idx = 4 * threadIdx.x; idx < (H + 2 * KVH) * half; idx += 4 * 256) {
        const int head = idx / half, i = idx - head * half;
        f32x4_t y0 = *reinterpret_cast<const f32x4_t *>(x + head * dh + i);
        f32x4_t y1 = *reinterpret_cast<const f32x4_t *>(x + head * dh + i + half);
        if (head < H + KVH) {
            const f32x4_t c01 = *reinterpret_cast<const f32x4_t *>(rope + (int64_t)pos * half + i);
            const f32x4_t c23 = *reinterpret_cast<const f32x4_t *>(rope + (int64_t)pos * half + i + 2);
            const float cx[4] = {c01[0], c01[2], c23[0], c23[2]}, cy[4] = {c01[1], c01[3], c23[1], c23[3]};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float r0 = y0[j] * cx[j] - y1[j] * cy[j];
                const float r1 = y1[j] * cx[j] + y0[j] * cy[j];
                y0[j] = r0;
                y1[j] = r1;
            }
        }
        if (head < H) {
            float *qo = q + (int64_t)m * H * dh + head * dh + i;
            *reinterpret_cast<f32x4_t *>(qo) = y0;
            *reinterpret_cast<f32x4_t *>(qo + half) = y1;
        } else {
            const bool is_k = head < H + KVH;
            const int g = is_k ? head - H : head - H - KVH;
            uint16_t *c = (is_k ? kc : vc) + (int64_t)g * stride + (int64_t)pos * dh + i;
            u32x2_t w0, w1;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                w0[j] = (uint32_t)bf16_rne_bits(y0[2 * j]) | ((uint32_t)bf16_rne_bits(y0[2 * j + 1]) << 16);
                w1[j] = (uint32_t)bf16_rne_bits(y1[2 * j]) | ((uint32_t)bf16_rne_bits(y1[2 * j + 1]) << 16);
            }
            *reinterpret_cast<u32x2_t *>(c) = w0;
            *reinterpret_cast<u32x2_t *>(c + half) = w1;
        }
    }
}

__global__ __launch_bounds__(256) void k_pf_swiglu_split(const float *gu, int F, uint16_t *out, int64_t out_term) {
    const int m = blockIdx.x;
    const float *x = gu + (int64_t)m * 2 * F;
    for (int f = 8 * threadIdx.x; f < F; f += 8 * 256) {
        float y[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float g = x[f + j], u = x[F + f + j];
            y[j] = g / (1.0f + expf(-g)) * u;
        }
        u32x4_t t[X_TERMS];
        split8(y, t);
#pragma unroll
        for (int i = 0; i < X_TERMS; ++i)
            *reinterpret_cast<u32x4_t *>(out + i * out_term + (int64_t)m * F + f) = t[i];
    }
}

}  // namespace

hipError_t launch_pf_embed(const uint16_t *emb, int d, const int32_t *tokens, int M, float *h, hipStream_t s) {
    hipLaunchKernelGGL(k_pf_embed, dim3(M), dim3(256), 0, s, emb, d, tokens, h);
    return hipGetLastError();
}

hipError_t launch_pf_norm_split(const float *h, int K, int M, const uint16_t *gain, float eps, uint16_t *out,
                                int64_t out_term, hipStream_t s) {
    if (K % 8)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_norm_split, dim3(M), dim3(256), 0, s, h, K, gain, eps, out, out_term);
    return hipGetLastError();
}

hipError_t launch_pf_fold_norm_split(float *h, const float *part, int splits, int K, int M, const uint16_t *gain,
                                     float eps, uint16_t *out, int64_t out_term, hipStream_t s) {
    if (K % 8 || splits < 1 || splits > PF_MAX_SPLITS)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_fold_norm_split, dim3(M), dim3(256), 0, s, h, part, splits, (int64_t)M * K, K, gain, eps,
                       out, out_term);
    return hipGetLastError();
}

hipError_t launch_pf_split_sum(const float *part, int splits, int64_t n, float *C, hipStream_t s) {
    if (splits < 1 || splits > PF_MAX_SPLITS || n < 1)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_split_sum, dim3((unsigned)std::min<int64_t>((n + 255) / 256, 4096)), dim3(256), 0, s, part,
                       splits, n, C, n);
    return hipGetLastError();
}

hipError_t launch_pf_gemm(const PfGemmArgs &a, int epi, hipStream_t s, int *fold) {
    if (fold)
        *fold = 0;
    if (a.M < 1 || a.N < 1 || a.K < 8 || a.K % 8 || a.lda % 8 || a.M > PF_ROWS)
        return hipErrorInvalidValue;
    if (epi == EPI_SWIGLU) {
        // gate/up: the SwiGLU in the wide kernel's epilogue when the launch
        // is wide (xout must not overlap A: other work-groups still read
        // it), else the product into C and a separate SwiGLU kernel.  Same
        // box, 13B prefill: 72.9 -> 72.4 ms.
        const int F = a.N / 2;
        if (a.N % 2 || F % 8 || !a.xout)
            return hipErrorInvalidValue;
        const int TMw = (a.M + GW_M - 1) / GW_M;
        const int t256 = TMw * ((F + 127) / 128), t224 = TMw * ((F + 111) / 112);
        if (t256 >= GW_MIN_TILES && a.K % GB_K == 0) {
            PfGemmArgs b = a;
            b.splits = 1;
            if ((int64_t)((t224 + 255) / 256) * 224 < (int64_t)((t256 + 255) / 256) * 256)
                hipLaunchKernelGGL((k_pf_gemm_wide<EPI_SWIGLU, 224>), dim3(8 * ((t224 + 7) / 8)), dim3(GW_THREADS), 0, s,
                                   b);
            else
                hipLaunchKernelGGL((k_pf_gemm_wide<EPI_SWIGLU, 256>), dim3(8 * ((t256 + 7) / 8)), dim3(GW_THREADS), 0, s,
                                   b);
            return hipGetLastError();
        }
        const hipError_t e = launch_pf_gemm(a, EPI_STORE, s);
        if (e != hipSuccess)
            return e;
        return launch_pf_swiglu_split(a.C, F, a.M, a.xout, a.x_term, s);
    }
    const int tiles = ((a.N + GB_N - 1) / GB_N) * ((a.M + GB_M - 1) / GB_M);
    // Wide layers (at least 128 tiles of 256 x 256) take the direct-to-LDS
    // kernel.  Both kernels fill the same fraction of the last round (one
    // 256 x 256 work-group per CU against two of 256 x 128); measured with
    // the 256 x 128 kernel's time first (us): 1023 rows, 13B QKV 509 -> 448,
    // gate/up 959 -> 857, 7B QKV 368 -> 335, 70B QKV 653 -> 599; 511 rows,
    // 7B gate/up 353 -> 311, 70B gate/up 1426 -> 1307.  With fewer tiles
    // (the QKV layers at 511 rows: 80-120 tiles) the 256 x 128 kernel stays
    // faster (13B 334 against 354).
    const int wide_tiles = ((a.N + GB_N - 1) / GB_N) * ((a.M + GW_M - 1) / GW_M);
    if (wide_tiles >= GW_MIN_TILES && a.K % GB_K == 0 && epi == EPI_STORE) {
        PfGemmArgs b = a;
        b.splits = 1;
        // Tiles 224 wide when that takes fewer tile-widths of rounds on 256
        // CUs: a round lasts about as long as a tile is wide, and 13B gate/up
        // (1023 rows) is 432 tiles of 256 (1.7 rounds) or 496 of 224 (1.9).
        const int tiles224 = ((a.N + 223) / 224) * ((a.M + GW_M - 1) / GW_M);
        const int64_t cost256 = (int64_t)((wide_tiles + 255) / 256) * 256;
        const int64_t cost224 = (int64_t)((tiles224 + 255) / 256) * 224;
        if (cost224 < cost256)
            hipLaunchKernelGGL((k_pf_gemm_wide<EPI_STORE, 224>), dim3(8 * ((tiles224 + 7) / 8)), dim3(GW_THREADS), 0, s,
                               b);
        else
            hipLaunchKernelGGL((k_pf_gemm_wide<EPI_STORE, 256>), dim3(8 * ((wide_tiles + 7) / 8)), dim3(GW_THREADS), 0,
                               s, b);
        return hipGetLastError();
    }
    // wide layers (at least one tile per CU): 4 x 2 waves, one stage in
    // flight; narrow ones: split residual updates (below), else 2 x 4 waves
    // with two stages in flight
    if (tiles >= 256) {
        PfGemmArgs b = a;
        b.splits = 1;
        const dim3 grid(8 * ((tiles + 7) / 8)), block(G_THREADS);
        if (epi == EPI_STORE)
            hipLaunchKernelGGL((k_pf_gemm<EPI_STORE, 4, 2, 1>), grid, block, 0, s, b);
        else if (epi == EPI_RESID)
            hipLaunchKernelGGL((k_pf_gemm<EPI_RESID, 4, 2, 1>), grid, block, 0, s, b);
        else
            return hipErrorInvalidValue;
        return hipGetLastError();
    }
    // Residual updates split the reduction over as many work-groups as fit
    // in one round: the 4 x 2-wave kernel runs two work-groups per CU, so up
    // to 512 (13B output and down projections: 160 tiles, 3 splits; at
    // least 16 stages per split).  Other narrow layers run unsplit.
    int splits = 1;
    bool wide_split = false;
    if (epi == EPI_RESID && a.part) {
        splits = std::min(PF_MAX_SPLITS, 512 / tiles);
        while (splits > 1 && a.K < splits * GB_K * 16)
            --splits;
        // The same split on 256 x 256 tiles (one work-group per CU) when it
        // keeps at least 160 CUs busy: 1023 rows, 13B O 185 -> 168 us, down
        // 462 -> 436; 511 rows, 70B O 221 -> 197, down 775 -> 684.  At the
        // 7B shape (511 rows, 128 work-groups) the 256 x 128 tiles stay
        // faster (O 76 against 86 us).
        int ws = std::min(PF_MAX_SPLITS, 256 / std::max(wide_tiles, 1));
        while (ws > 1 && a.K < ws * GB_K * 16)
            --ws;
        if (a.K % GB_K == 0 && ws > 1 && wide_tiles * ws >= GW_MIN_SPLIT_GROUPS) {
            splits = ws;
            wide_split = true;
        }
    }
    PfGemmArgs b = a;
    b.splits = splits;
    const dim3 grid(8 * ((tiles * b.splits + 7) / 8)), block(G_THREADS);
    if (splits > 1) {
        if (wide_split)
            hipLaunchKernelGGL((k_pf_gemm_wide<EPI_PARTIAL, 256>), dim3(8 * ((wide_tiles * splits + 7) / 8)),
                               dim3(GW_THREADS), 0, s, b);
        else
            hipLaunchKernelGGL((k_pf_gemm<EPI_PARTIAL, 4, 2, 1>), grid, block, 0, s, b);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        if (fold && a.ldc == a.N) {
            *fold = splits;  // the next norm adds the partials
            return hipSuccess;
        }
        return launch_pf_split_sum(a.part, splits, (int64_t)a.M * a.ldc, a.C, s);
    } else if (epi == EPI_STORE) {
        hipLaunchKernelGGL((k_pf_gemm<EPI_STORE, 2, 4, 2>), grid, block, 0, s, b);
    } else if (epi == EPI_RESID) {
        hipLaunchKernelGGL((k_pf_gemm<EPI_RESID, 2, 4, 2>), grid, block, 0, s, b);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_pf_rope_kv(const float *qkv, int M, int start, const float2 *rope, int H, int KVH, int dh,
                             float *q, uint16_t *kcache, uint16_t *vcache, int64_t kv_head_stride, hipStream_t s) {
    if (dh % 8 || kv_head_stride % 4)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_rope_kv, dim3(M), dim3(256), 0, s, qkv, start, rope, H, KVH, dh, q, kcache, vcache,
                       kv_head_stride);
    return hipGetLastError();
}

hipError_t launch_pf_attention(const PfAttnArgs &a, hipStream_t s) {
    if (a.M < 1 || a.n_heads < 1 || a.n_kv_heads < 1 || a.n_heads % a.n_kv_heads)
        return hipErrorInvalidValue;
    const dim3 grid(((a.M + 63) / 64) * a.n_heads), block(256);
    switch (a.head_dim) {
    case 32:
        hipLaunchKernelGGL(k_pf_attn<32>, grid, block, 0, s, a);
        break;
    case 64:
        hipLaunchKernelGGL(k_pf_attn<64>, grid, block, 0, s, a);
        break;
    case 128:
        hipLaunchKernelGGL(k_pf_attn<128>, grid, block, 0, s, a);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_pf_swiglu_split(const float *gu, int F, int M, uint16_t *out, int64_t out_term, hipStream_t s) {
    if (F % 8)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_pf_swiglu_split, dim3(M), dim3(256), 0, s, gu, F, out, out_term);
    return hipGetLastError();
}

}  // namespace sdk
