// Library-internal declarations shared by the HIP kernels and the host
// orchestration.  Not part of the public ABI (include/sd.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sdk {

// Rows of one forward: the verification of K_max <= 15 drafts plus the last
// committed token, one 16-row MFMA tile, and the prefill chunk size.
constexpr int MAX_ROWS = 16;
// Keys per attention work-group (split-KV chunk): 128 for the matrix-core
// and float32 kernels, 64 for the VALU kernel of one or two query vectors
// per kv head (two waves of 32 keys).
constexpr int ATTN_CHUNK = 128;
constexpr int ATTN_CHUNK_VALU = 64;
// Largest head_dim the attention kernel stages in LDS.
constexpr int MAX_HEAD_DIM = 128;
// Longest context (cache capacity) and the most key chunks one attention
// call combines: 65536 positions in 64-key chunks.
constexpr int MAX_CONTEXT = 65536;
constexpr int MAX_SPLITS = MAX_CONTEXT / ATTN_CHUNK_VALU;
// Keys per chunk of the finest split a model's attention can take: 64 when
// it can run the VALU kernel (bfloat16, head_dim 128, at most two query
// heads per kv head), else 128; and the split partial slots a cache of
// capacity cap then needs.
__host__ __device__ constexpr int attn_chunk_min(bool bf16, int head_dim, int n_heads, int n_kv_heads) {
    return (bf16 && head_dim == 128 && n_heads <= 2 * n_kv_heads) ? ATTN_CHUNK_VALU : ATTN_CHUNK;
}
__host__ __device__ constexpr int attn_split_slots(int cap, int chunk_min) { return (cap + chunk_min - 1) / chunk_min; }

// Where and what the current forward computes.  Device resident: the
// greedy head of one step writes the control block of the next step, so
// the host never needs token ids or positions during decoding.
struct DevCtl {
    int32_t pos;               // position of row 0
    int32_t m;                 // rows in this forward, 1..MAX_ROWS; 0: a cancelled step (every kernel returns)
    int32_t tokens[MAX_ROWS];  // input token of every row
    int32_t m_next;            // self-speculative decoding: rows of the next step, set by the decision
};

enum Phase : int32_t { PHASE_DRAFT = 0, PHASE_VERIFY = 1 };

// Decoding state of one generate call (device resident).
struct DevState {
    int32_t lc;        // committed KV length: the cache holds every committed token but the last
    int32_t last;      // last committed token, input of the next forward
    int32_t emitted;   // tokens written to out_tokens
    int32_t max_new;
    int32_t k;         // drafts of the current stage so far
    int32_t kcap;      // draft budget of the current stage
    int32_t k_max;
    int32_t phase;     // what the next step is
    int32_t gen_done;
    int32_t seq;       // steps finished (mirrors the mailbox)
    float gamma;       // draft-exit threshold of the current stage
    int32_t adaptive;  // 1: gamma follows the adaptive rule after each verification
    int32_t n_updates; // stages that updated the threshold
    int32_t pad;
    double ar;         // smoothed acceptance rate
    double gamma_d;    // threshold in float64; gamma is its float32 rounding
    double alpha, epsilon, beta1, beta2;
    int32_t drafts[MAX_ROWS];
    float dpmax[MAX_ROWS];
    int64_t n_stages, n_drafted, n_accepted, n_draft_steps;
    uint64_t dqw[MAX_ROWS];  // sampling: fixed-point weight of each draft under its draft distribution
};

// Pinned host memory the GPU writes after every self-speculative step: one
// 64-bit word (step sequence number in bits 0-31, phase in 32-35, the
// generation-done flag in bit 36, tokens emitted in 40-63), written by a
// single relaxed store, so the host never sees a torn state and the GPU
// needs no release fence (which would write back the whole L2).
struct Mailbox {
    uint64_t word;
};

__host__ __device__ inline uint64_t mb_pack(int32_t seq, int32_t phase, int32_t gen_done, int32_t emitted) {
    return (uint64_t)(uint32_t)seq | ((uint64_t)(phase & 15) << 32) | ((uint64_t)(gen_done & 1) << 36) |
           ((uint64_t)(emitted & 0xffffff) << 40);
}
__host__ __device__ inline int32_t mb_seq(uint64_t w) { return (int32_t)(uint32_t)(w & 0xffffffffu); }
__host__ __device__ inline int32_t mb_phase(uint64_t w) { return (int32_t)((w >> 32) & 15); }
__host__ __device__ inline bool mb_done(uint64_t w) { return ((w >> 36) & 1) != 0; }
__host__ __device__ inline int32_t mb_emitted(uint64_t w) { return (int32_t)((w >> 40) & 0xffffff); }

enum HeadMode : int32_t { HEAD_NONE = 0, HEAD_AR = 1, HEAD_DRAFT = 2, HEAD_VERIFY = 3 };

// EPI_PARTIAL: split-K partial sums [split][row][N], folded into the
// residual stream by the next k_prep_norm (MFMA path only).
enum Epi : int { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_HEAD = 4, EPI_PARTIAL = 5 };

// Activations of the MFMA path: a float32 value u is held as X_TERMS
// bfloat16 terms hi + mid + lo, each the round-to-nearest-even of what the
// previous terms leave; the remainders are exact in float32, so the three
// terms reproduce every normal float32 value exactly.  A two-term split
// (about 17 bits) lets the few-ulp differences it leaves in K/V flip their
// bfloat16 rounding in the cache, and the flips compound with depth.
constexpr int X_TERMS = 3;

__device__ __forceinline__ uint16_t bf16_rne_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// MFMAs per k-step (16 packed columns each) for up to max_rows rows.
__host__ __device__ constexpr int mfma_packs(int max_rows) { return (X_TERMS * max_rows + 15) / 16; }

// MFMA work-group shape (16-row tiles per work-group, waves per work-group)
// by output kind and packing count, from sweeps at the 13B shapes: two
// tiles for the split-K output projections, four otherwise (at 4, 8 and 13
// rows); four waves throughout.  The launcher takes eight tiles for wide
// gate/up and lm-head layers at three packings (launch_mfma_np).
__host__ __device__ constexpr int mfma_shape_tn(int epi, int np) {
    return (void)np, epi == EPI_PARTIAL ? 2 : 4;
}
__host__ __device__ constexpr int mfma_shape_nw(int epi, int np) { return (void)epi, (void)np, 4; }

// Fragment layout of the MFMA-path activations.  For k-step q = k / 128,
// packing p and 32-wide slice i = (k % 128) / 32, the 16 columns x 32 k of
// one MFMA B operand are 512 contiguous bf16 in lane order: lane
// column + 16 ((k % 32) / 8) holds 8 consecutive k.  Column c = t M + r
// carries term t of row r (M rows in this forward).  X_PACKS_MAX packings
// are reserved per k-step, so a buffer holds 48 K elements for any M, and
// an MFMA operand is one coalesced 1 KB load.
constexpr int X_PACKS_MAX = 3;
__host__ __device__ inline int64_t xfrag_off(int t, int r, int k, int M) {
    const int c = t * M + r, p = c >> 4, lane = (c & 15) + 16 * ((k & 31) >> 3);
    return ((((int64_t)(k >> 7) * X_PACKS_MAX + p) * 4 + ((k & 127) >> 5)) << 9) + lane * 8 + (k & 7);
}

// Splits u into X_TERMS bf16 terms.
__device__ __forceinline__ void split3(float u, uint16_t (&t)[X_TERMS]) {
    t[0] = bf16_rne_bits(u);
    const float r1 = u - __uint_as_float((uint32_t)t[0] << 16);
    t[1] = bf16_rne_bits(r1);
    t[2] = bf16_rne_bits(r1 - __uint_as_float((uint32_t)t[1] << 16));
}

// Stores the terms of activation (row r, index k) of an M-row forward.
__device__ __forceinline__ void store_split3(uint16_t *x, int r, int k, int M, float u) {
    uint16_t t[X_TERMS];
    split3(u, t);
#pragma unroll
    for (int i = 0; i < X_TERMS; ++i)
        x[xfrag_off(i, r, k, M)] = t[i];
}

struct HeadArgs {
    int32_t mode;
    float *logits;       // optional float32 [m][ld_logits]
    int64_t ld_logits;
    float4 *partials;    // [n_tiles][MAX_ROWS]: (max, argmax bits, sum exp(l - max), 0)
    DevState *st;
    Mailbox *mb;         // device view of the pinned mailbox (HEAD_DRAFT / HEAD_VERIFY)
    int32_t *out_tokens;
    int32_t *stage_log;  // [stage_log_cap][2]
    float *gamma_log;    // [stage_log_cap]: threshold each stage drafted with
    int32_t stage_log_cap;
    int32_t logits_by_draft;  // sampling drafts: the (one-row) logits go to row st->k of logits
    int32_t sampled;          // sampling variant: the sampling kernels take the decision
};

// ---------------------------------------------------------------------------
// Sampling variant.  The warped distribution of a row of logits l is
// w_x = exp((l_x - max l) / T) restricted to its top-p nucleus: the shortest
// prefix of the tokens in (w descending, id ascending) order whose mass
// reaches top_p.  Masses are fixed point, W_x = trunc(w_x 2^31) (at most
// 2^31, as w_x <= 1), summed in uint64, so every sum, cut and cumulative
// mass is exact and independent of the summation order.  The nucleus is
// {w_x > w*} plus the first n_tie tokens (by id) with w_x == w*.
constexpr float WFIX = 2147483648.0f;  // 2^31

struct SampleParams {
    float temperature;
    float top_p;
    uint64_t seed;
};

struct RowStat {
    float mx;         // max logit of the row
    uint32_t bstar;   // bit pattern of w*
    uint32_t n_tie;   // tokens with w == w* in the nucleus, lowest ids first
    uint32_t pad;
    uint64_t zs;      // nucleus mass
    uint64_t wd;      // verification row r: weight of draft r + 1 if in the nucleus, else 0
};

// Purposes of the uniforms: the second counter word of Philox4x64-10, whose
// counter is (output index, purpose, stage, 0) and key (seed, 0).
enum UniformPurpose : int32_t { U_DRAFT = 0, U_ACCEPT = 1, U_FINAL = 2 };

struct SampleArgs {
    SampleParams sp;
    int32_t vocab;
    const DevCtl *ctl;
    const float *vlog;  // [MAX_ROWS][vocab]: logits of the verification or autoregressive rows
    const float *dlog;  // [MAX_ROWS][vocab]: logits of the drafts of the stage, by draft index
    RowStat *vstat;     // [MAX_ROWS]
    RowStat *dstat;     // [MAX_ROWS]
    HeadArgs head;
};

struct EpiArgs {
    float *out;            // STORE/RESID: [m][ld_out]; SWIGLU: [m][ffn]
    int64_t ld_out;
    uint16_t *out_x;       // SWIGLU: when set, the output split into bf16 terms in fragment layout (xfrag_off)
    float *q;              // QKV: rotated queries [m][n_heads * head_dim]
    int64_t ld_q;
    void *kcache, *vcache; // QKV: this layer's K and V: [n_kv_heads][cap][head_dim]
    int64_t kv_head_stride;
    const float2 *rope;    // [positions][head_dim / 2] of (cos, sin)
    int32_t n_heads, n_kv_heads, head_dim, ffn;
    HeadArgs head;
};

struct LinearArgs {
    const void *W;         // [N][K] row-major, weight dtype
    int32_t N, K;
    const float *X;        // VALU paths: activations [m][ldx] float32
    const uint16_t *Xs;    // MFMA path: activations split into bf16 terms in fragment layout (xfrag_off)
    int32_t max_rows;      // MFMA path: host bound on ctl->m, sets the MFMAs per k-step
    int64_t ldx;
    const void *gain;      // VALU paths: RMSNorm gain [K] (weight dtype), or null: no norm
    const float *ssq;      // MFMA path with RMSNorm: the slices' sums of h^2 [MAX_ROWS][ssq_slices]
                           // (the fragments then hold gain * h), or null: no norm
    int32_t ssq_slices;
    float eps;
    const DevCtl *ctl;
    EpiArgs epi;
    int32_t waves;         // MFMA path: waves per work-group splitting the reduction
    int32_t splits;        // EPI_PARTIAL: work-groups splitting the reduction per tile group
    float *part;           // EPI_PARTIAL: [splits][MAX_ROWS][N]
    int32_t n_tiles;       // tiles in the layer (set by launch_linear)
    const int32_t *wexp;   // PATH_GEMV_FP8: per weight row, the exponent e of its 2^e scale
    int32_t guarded;       // part of a step enqueued ahead, which the step guard may cancel (ctl->m = 0):
                           // the one-row path then takes its row count from ctl->m too
};

struct AttnArgs {
    const float *q;        // [m][n_heads * head_dim]
    int64_t ld_q;
    const void *kcache, *vcache;  // this layer: [n_kv_heads][cap][head_dim]
    int64_t kv_head_stride;
    float *part_o;         // [splits][n_heads][MAX_ROWS][head_dim]
    float2 *part_ml;       // [splits][n_heads][MAX_ROWS]: (running max, sum of exp)
    float *out;            // [m][n_heads * head_dim]
    uint16_t *out_x;       // when set, the output split into bf16 terms in fragment layout instead
    int64_t ld_out;
    int32_t n_heads, n_kv_heads, head_dim;
    int32_t cap;           // cache capacity: positions past it are never read
    int32_t splits, chunk; // set by launch_attention: key chunks and keys per chunk
    const DevCtl *ctl;
};

// ---------------------------------------------------------------------------
// Large-M forward (prompt prefill, long forwards): up to PF_ROWS rows at
// positions [start, start + M), bfloat16 weights and KV.  Activations that
// feed a matrix-core GEMM are held as X_TERMS bf16 terms, row-major:
// [X_TERMS][PF_ROWS][ld] with the term stride PF_ROWS * ld.
constexpr int PF_ROWS = 1024;
constexpr int PF_MAX_SPLITS = 4;  // k-splits of a narrow residual-update GEMM

// C[m][n] = (EPI_STORE) or += (EPI_RESID) sum over the terms t of
// A_t[m][0..K) . W[n][0..K).
struct PfGemmArgs {
    const uint16_t *W;  // [N][K] bf16
    const uint16_t *A;  // [X_TERMS][.][lda] bf16 terms, M rows used
    int64_t a_term;     // elements between terms
    float *C;           // [M][ldc]
    int64_t ldc;
    int32_t M, N, K, lda;
    float *part;        // EPI_RESID: [PF_MAX_SPLITS][M][ldc] scratch for a split reduction, or null
    int32_t splits;     // set by the launcher
    // EPI_SWIGLU (W = [gate; up], N = 2 F): silu(gate) * up as X_TERMS bf16
    // terms into xout [X_TERMS][.][F] (term stride x_term); C [M][2 F] is
    // scratch for shapes the fused kernel does not take
    uint16_t *xout;
    int64_t x_term;
};

// Causal attention of M query rows (row m at position start + m) over the
// cached keys [0, start + m], output written as X_TERMS bf16 terms.
struct PfAttnArgs {
    const float *q;  // [M][ldq] rotated queries
    int64_t ldq;
    const uint16_t *kcache, *vcache;  // this layer: [n_kv_heads][cap][head_dim]
    int64_t kv_head_stride;
    uint16_t *out;  // [X_TERMS][.][ldo]
    int64_t out_term, ldo;
    int32_t M, start, n_heads, n_kv_heads, head_dim;
};

hipError_t launch_pf_embed(const uint16_t *emb, int d, const int32_t *tokens, int M, float *h, hipStream_t s);
// g * h / rms(h) of every row (g: gain [K] bf16), as X_TERMS terms into out.
hipError_t launch_pf_norm_split(const float *h, int K, int M, const uint16_t *gain, float eps, uint16_t *out,
                                int64_t out_term, hipStream_t s);
// The same after folding split-K partials into h: h[m] += part[0][m] +
// part[1][m] + ... (splits of them, [splits][M][K], in split order) first.
hipError_t launch_pf_fold_norm_split(float *h, const float *part, int splits, int K, int M, const uint16_t *gain,
                                     float eps, uint16_t *out, int64_t out_term, hipStream_t s);
// C = A W^T (EPI_STORE), C += A W^T (EPI_RESID), or the SwiGLU of a gate/up
// product as terms (EPI_SWIGLU, see PfGemmArgs).  A narrow EPI_RESID may
// split its reduction into a.part; with fold null the partials are added
// into C before the call returns (on the stream), else *fold receives the
// number of splits left in a.part for launch_pf_fold_norm_split (0: none).
hipError_t launch_pf_gemm(const PfGemmArgs &a, int epi, hipStream_t s, int *fold = nullptr);
// C[i] += part[0][i] + part[1][i] + ... for i < n (part [splits][n]).
hipError_t launch_pf_split_sum(const float *part, int splits, int64_t n, float *C, hipStream_t s);
// Rotary embedding of q and k from the QKV GEMM output [M][(H + 2 KVH) dh];
// q into q [M][H dh], k and v into the cache at positions start + m.
hipError_t launch_pf_rope_kv(const float *qkv, int M, int start, const float2 *rope, int H, int KVH, int dh,
                             float *q, uint16_t *kcache, uint16_t *vcache, int64_t kv_head_stride, hipStream_t s);
hipError_t launch_pf_attention(const PfAttnArgs &a, hipStream_t s);
// silu(gate) * up of the gate/up GEMM output [M][2 F], as X_TERMS terms.
hipError_t launch_pf_swiglu_split(const float *gu, int F, int M, uint16_t *out, int64_t out_term, hipStream_t s);

// Kernel paths of the linear layers.
// PATH_WAVE2: up to two rows on one-wave tiles (bf16 weights).
// PATH_GEMV_FP8: one row over the draft's FP8 weights (LinearArgs::wexp).
enum LinearPath : int { PATH_GEMV = 0, PATH_VALU16 = 1, PATH_MFMA = 2, PATH_VALU2 = 3, PATH_WAVE2 = 4,
                        PATH_GEMV_FP8 = 5 };

// Optional events the runtime records at a launch's own start and end.
struct LaunchTiming {
    hipEvent_t start = nullptr, stop = nullptr;
};

// Host-side launchers (kernels_*.hip).  bf16 selects bfloat16 weights and KV.
// chunks: PATH_WAVE2 loads in flight per wave (1 or 2; 0: two for 4 weight
// rows, one for 8).
hipError_t launch_linear(const LinearArgs &a, int epi, bool bf16, int path, int rows_per_tile, int n_tiles,
                         hipStream_t s, const LaunchTiming &t = LaunchTiming{}, int chunks = 0);
// PATH_WAVE2 loads in flight for a tile of `rows` weight rows when the plan
// leaves it open.
constexpr int wave2_default_chunks(int rows) { return rows == 4 ? 2 : 1; }
// FP8 E4M3 copy of a bf16 matrix [N][K]: bytes Q [N][K] and the exponent of
// each row's power-of-two scale E [N] (see k_quantize_fp8).
hipError_t launch_quantize_fp8(const uint16_t *W, int32_t N, int32_t K, uint8_t *Q, int32_t *E, hipStream_t s);
// Elements per work-group of the MFMA-path input preparation.
constexpr int PREP_SLICE = 512;
__host__ __device__ constexpr int prep_slices(int K) { return (K + PREP_SLICE - 1) / PREP_SLICE; }
// g * h, or plain h (gain == null), split into X_TERMS bf16 terms in fragment
// layout for the MFMA path (K a multiple of 128), with the sums of h^2 of
// each PREP_SLICE-element slice in ssq [MAX_ROWS][prep_slices(K)] (gain set)
// for the consumer's 1/rms(h).  First adds n_part pending split-K partials
// ([n_part][MAX_ROWS][K]) into h.
hipError_t launch_prep_norm(float *h, int64_t ldh, const void *gain, bool bf16, int K, const DevCtl *ctl,
                            uint16_t *xs, const float *part, int n_part, float *ssq, hipStream_t s);
// After a head linear: combines its n_tiles partials and takes the decoding decision.
hipError_t launch_head_finalize(const LinearArgs &a, int n_tiles, hipStream_t s);
// Sampling variant, after a head linear that wrote the logits: the nucleus
// statistics of every row (one work-group per row, up to max_rows), then the
// decision of the step in one work-group (draw, acceptance, state update).
hipError_t launch_sample_step(const SampleArgs &a, int max_rows, hipStream_t s);
constexpr int32_t MAX_SAMPLE_VOCAB = 524288;  // largest vocabulary the sampling kernels take
hipError_t launch_attention(const AttnArgs &a, bool bf16, int max_rows, hipStream_t s);
hipError_t launch_embed(const void *emb, bool bf16, int d, const DevCtl *ctl, float *h, int64_t ldh,
                        hipStream_t s);
hipError_t launch_set_ctl(DevCtl *ctl, int32_t pos, int32_t m, const int32_t *dev_tokens, hipStream_t s);
// The same from m <= MAX_ROWS host tokens, passed as a kernel argument.
hipError_t launch_set_ctl_host(DevCtl *ctl, int32_t pos, int32_t m, const int32_t *host_tokens, hipStream_t s);
// Threshold rule of a generate call: fixed gamma (adaptive = 0) or the
// adaptive rule starting at gamma0.
struct ExitRule {
    int32_t adaptive;
    float gamma;
    double gamma0, alpha, epsilon, beta1, beta2;
};
// First kernel of a self-speculative step the host enqueued as (phase,
// max_rows): the step runs (ctl->m = ctl->m_next) when the device's decision
// asks for that kind of step, else it is cancelled (ctl->m = 0).
hipError_t launch_step_guard(DevCtl *ctl, const DevState *st, int32_t phase, int32_t max_rows, hipStream_t s);
hipError_t launch_init_decode(DevState *st, DevCtl *ctl, Mailbox *mb, int32_t lc, const int32_t *dev_last,
                              int32_t max_new, int32_t k_max, const ExitRule &rule, hipStream_t s);
hipError_t launch_fill_zero(void *p, size_t bytes, hipStream_t s);

// ---------------------------------------------------------------------------
// Wave sums of several values at once, on the VALU.  A butterfly over the
// lane bits 5, 4, 3, 2 halves the number of values at each level: a lane
// keeps the half of its values that the lane bit selects and adds its
// partner's copy of the same half (the pair of lanes 32 and 16 apart swaps
// halves with one v_permlane32_swap / v_permlane16_swap, the pair 8 apart
// exchanges through a row rotation, the pair 4 apart through a half-row
// mirror), then the four lanes of a quad add up by two quad permutations.
// After that, value j's total is in the lanes whose bits 5, 4, 3, 2 spell
// j's bits 0, 1, 2, 3 (all four lanes of the quad): 15 swaps or moves and
// 15 adds for 16 values, against 96 shuffles through LDS (ds_bpermute) one
// at a time.  A level with a single value left adds the partner's copy.
// The order of the additions is fixed, so sums are deterministic.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int DPP_ROW_ROR8 = 0x128;
constexpr int DPP_ROW_HALF_MIRROR = 0x141;
constexpr int DPP_QUAD_XOR2 = 0x4e;  // quad_perm [2, 3, 0, 1]
constexpr int DPP_QUAD_XOR1 = 0xb1;  // quad_perm [1, 0, 3, 2]

// lanes 0-31 get a's sum over lanes l and l + 32, lanes 32-63 b's
__device__ __forceinline__ float bfly32(float a, float b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// rows 0 and 2 (lanes 0-15, 32-47) get a's sum over rows 2i, 2i + 1, rows 1 and 3 b's
__device__ __forceinline__ float bfly16(float a, float b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// lanes with bit 3 clear get a's sum over lanes l and l ^ 8, the others b's
__device__ __forceinline__ float bfly8(float a, float b, int lane) {
    const bool hi = lane & 8;
    return (hi ? b : a) + dpp_mov<DPP_ROW_ROR8>(hi ? a : b);
}
// lanes with bit 2 clear get a's sum over lanes l and the mirror 7 - l of the half row, the others b's
__device__ __forceinline__ float bfly4(float a, float b, int lane) {
    const bool hi = lane & 4;
    return (hi ? b : a) + dpp_mov<DPP_ROW_HALF_MIRROR>(hi ? a : b);
}

// lanes with bit 1 clear get a's sum over lanes l and l ^ 2, the others b's
__device__ __forceinline__ float bfly2(float a, float b, int lane) {
    const bool hi = lane & 2;
    return (hi ? b : a) + dpp_mov<DPP_QUAD_XOR2>(hi ? a : b);
}

// Totals over the wave of v[0..N) (N a power of two, at most 16), returned
// per lane as described above; wave_sums_lane(j) is the first lane holding j.
template <int N>
__device__ __forceinline__ float wave_sums(const float (&v)[N], int lane) {
    static_assert(N >= 1 && N <= 16 && (N & (N - 1)) == 0, "1, 2, 4, 8 or 16 values");
    float a[16];
#pragma unroll
    for (int j = 0; j < N; ++j)
        a[j] = v[j];
    // value index bits, low first, follow lane bits 5, 4, 3, 2
    constexpr int n1 = N >= 2 ? N / 2 : 1;
#pragma unroll
    for (int j = 0; j < n1; ++j)
        a[j] = N >= 2 ? bfly32(a[2 * j], a[2 * j + 1]) : bfly32(a[0], a[0]);
    constexpr int n2 = n1 >= 2 ? n1 / 2 : 1;
#pragma unroll
    for (int j = 0; j < n2; ++j)
        a[j] = n1 >= 2 ? bfly16(a[2 * j], a[2 * j + 1]) : bfly16(a[0], a[0]);
    constexpr int n3 = n2 >= 2 ? n2 / 2 : 1;
#pragma unroll
    for (int j = 0; j < n3; ++j)
        a[j] = n2 >= 2 ? bfly8(a[2 * j], a[2 * j + 1], lane) : a[0] + dpp_mov<DPP_ROW_ROR8>(a[0]);
    float t = n3 >= 2 ? bfly4(a[0], a[1], lane) : a[0] + dpp_mov<DPP_ROW_HALF_MIRROR>(a[0]);
    t += dpp_mov<DPP_QUAD_XOR2>(t);
    t += dpp_mov<DPP_QUAD_XOR1>(t);
    return t;
}
__host__ __device__ constexpr int wave_sums_lane(int j) {
    return 32 * (j & 1) + 16 * ((j >> 1) & 1) + 8 * ((j >> 2) & 1) + 4 * ((j >> 3) & 1);
}
// the value index a lane holds (for the lanes wave_sums_lane names)
__device__ __forceinline__ int wave_sums_index(int lane) {
    return ((lane >> 5) & 1) | (((lane >> 4) & 1) << 1) | (((lane >> 3) & 1) << 2) | (((lane >> 2) & 1) << 3);
}


// Whole-wave max and sum with every lane receiving the result, on the VALU
// (the same lane exchanges as wave_sums, each level combining a lane with
// its partner's copy).
__device__ __forceinline__ float wave_max_all(float v) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    v = fmaxf(v, dpp_mov<DPP_ROW_ROR8>(v));
    v = fmaxf(v, dpp_mov<DPP_ROW_HALF_MIRROR>(v));
    v = fmaxf(v, dpp_mov<DPP_QUAD_XOR2>(v));
    return fmaxf(v, dpp_mov<DPP_QUAD_XOR1>(v));
}
__device__ __forceinline__ float wave_sum_all(float v) {
    const float a[1] = {v};
    return wave_sums<1>(a, 0);
}

}  // namespace sdk
