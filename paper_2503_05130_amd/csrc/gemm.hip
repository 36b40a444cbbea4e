// bf16 MFMA GEMM with fused epilogues for gfx950 (CDNA4).
//
// out[t, f] = epilogue( sum_k A[t, k] * W[f, k] + bias[f] )
//   A: activations, bf16 [M, K] row-major (tokens x features-in)
//   W: weights stored output-major, bf16 [N, K] row-major
//
// Data movement.  K is walked in 64-wide tiles.  Each tile of A and W is copied
// from global memory straight into LDS with global_load_lds_dwordx4 (gfx950's
// 16-byte global->LDS DMA: no VGPR staging), into an S-stage ring, so S-1
// tiles are in flight while one is consumed.  Each wave copies whole 8-row
// groups (one 1 KB DMA per group); LDS rows are 128 bytes with the 16-byte
// chunks XOR-swizzled per row, chosen so that the 16 rows read by one
// ds_read_b128 fragment load fall in distinct bank groups.  The swizzle is
// applied on the source side: lane i of a DMA fetches the global chunk that
// belongs at its fixed LDS slot.  The wave waits for its own DMAs of the tile
// it is about to read (s_waitcnt vmcnt), then a workgroup barrier makes every
// wave's copies visible and frees the slot the next DMA will overwrite.
//
// Math.  v_mfma_f32_16x16x32_bf16 on C^T blocks (features x tokens): the W
// fragment is the MFMA "A" operand, the activation fragment the "B" operand,
// so each lane ends up owning 4 consecutive output features of one token and
// stores them with one vector store.  4 waves in a 2 x 2 grid over the tile.
//
// Determinism and batch invariance: every configuration uses the same MFMA
// instruction; the K summation order (sequential 64-wide K tiles, or the
// workgroup-internal even/odd split for long K) is a function of the weight
// shape (N, K) alone.  So out[t, f] depends only on row t of A and row f of W
// -- never on the tile shape, the ring depth, the grid, the CU mask or the
// other rows in the batch.  No atomics, no cross-workgroup split-K.
#include "kernels.h"

#include <algorithm>

namespace iefwd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void *lds_ptr_t;

constexpr int kBK = 64;               // K tile (bf16 elements) = one 128-byte LDS row
constexpr int kThreads = 256;         // 4 waves in a 2 x 2 grid over the tile

struct GemmParams {
    const bf16_t *a;
    const bf16_t *w;
    const bf16_t *bias;
    const float *resid;
    void *out;
    int M, N, K;
    int tiles_m, tiles_n;
    QkvDst qkv;
    LnResid ln;
};

// Workgroups are dispatched round-robin over the 8 XCDs.  Renumber them so
// that each XCD receives a contiguous range of logical tiles (bijective for
// any grid size), which keeps tiles that share operands in one XCD's L2.
__device__ inline int xcd_contiguous(int i, int g) {
    constexpr int X = 8;
    const int q = g / X, r = g % X;
    const int x = i % X, local = i / X;
    return x < r ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

// Logical tile -> (token tile, feature tile), grouped 4 token tiles deep so
// that workgroups running together share both A rows and W rows.
__device__ inline void grouped_tile(int l, int tiles_m, int tiles_n, int &tm, int &tn) {
    constexpr int G = 4;
    const int per_group = G * tiles_n;
    const int g = l / per_group;
    const int first = g * G;
    const int gsize = min(tiles_m - first, G);
    const int in = l - g * per_group;
    tm = first + in % gsize;
    tn = in / gsize;
}


__device__ inline bf16_t f32_to_bf16(float f) {
    __bf16 b = (__bf16)f;   // round to nearest even
    return __builtin_bit_cast(bf16_t, b);
}

__device__ inline uint32_t pack2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// GELU(u) = u/2 (1 + erf(u / sqrt 2)), with erf from Abramowitz & Stegun,
// Handbook of Mathematical Functions, formula 7.1.26 (|error| <= 1.5e-7 for
// x >= 0): erfc(x) ~= (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),
// t = 1 / (1 + p x).  Written through erfc so that u < 0 keeps its relative
// accuracy: GELU(u) = u (1 - erfc(x)/2) for u >= 0 and u erfc(x)/2 for u < 0,
// x = |u| / sqrt 2.  About 14 VALU operations instead of a full erff.
__device__ inline float gelu(float u) {
    const float x = fabsf(u) * 0.7071067811865476f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
    float poly = fmaf(1.061405429f, t, -1.453152027f);
    poly = fmaf(poly, t, 1.421413741f);
    poly = fmaf(poly, t, -0.284496736f);
    poly = fmaf(poly, t, 0.254829592f);
    const float erfc_x = poly * t * __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
    return u * (u >= 0.f ? fmaf(-0.5f, erfc_x, 1.0f) : 0.5f * erfc_x);
}

// 16-byte chunk position of logical chunk 0 in LDS row r (row r holds its
// chunk c at position c ^ swizzle(r)).  Consecutive rows alternate between the
// two 128-byte halves of a 256-byte bank line, and within each parity the 8
// rows of a 16-row fragment get 8 distinct positions.
__device__ inline int swizzle(int r) { return ((r >> 1) & 7) ^ ((r & 1) << 2); }

// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (expcnt and lgkmcnt left unconstrained).
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// One 4-wave group's main loop over the K tiles kt_first, kt_first + kt_stride,
// ... (n_mine of them) through its own S-slot LDS ring, accumulating into acc.
// Every wave of the workgroup runs n_steps iterations (>= n_mine), so the
// workgroup barriers line up even when two groups own different tile counts.
template <int BM, int BN, int S>
__device__ inline void main_loop(const GemmParams &p, bf16_t *ring0, int wave, int lane, int m0, int n0,
                                 int kt_first, int kt_stride, int n_mine, int n_steps,
                                 f32x4 (&acc)[BN / 32][BM / 32]) {
    constexpr int TM = BM / 2, TN = BN / 2;          // per-wave tile (tokens x features)
    constexpr int FM = TM / 16, FN = TN / 16;        // 16x16 MFMA blocks per wave
    constexpr int STAGE = (BM + BN) * kBK;           // bf16 elements per ring slot
    constexpr int A_PW = BM / 32, W_PW = BN / 32;    // 1 KB DMAs per wave per K tile
    constexpr int LPW = A_PW + W_PW;
    static_assert(BM % 32 == 0 && BN % 32 == 0, "tile");
    static_assert(S >= 2 && (S - 2) * LPW <= 63, "ring depth");
    const int wm = wave >> 1, wn = wave & 1;

    // DMA sources of this lane: DMA i of this wave copies the 8-row group
    // g = wave + 4 i; lane l fills row 8 g + l / 8 at chunk position l % 8.
    // Rows past M / N are clamped to the last valid row (never stored).
    uint32_t a_src[A_PW], w_src[W_PW];
#pragma unroll
    for (int i = 0; i < A_PW; ++i) {
        const int r = 8 * (wave + 4 * i) + (lane >> 3);
        a_src[i] = (uint32_t)min(m0 + r, p.M - 1) * (uint32_t)p.K + (((lane & 7) ^ swizzle(r)) * 8);
    }
#pragma unroll
    for (int i = 0; i < W_PW; ++i) {
        const int r = 8 * (wave + 4 * i) + (lane >> 3);
        w_src[i] = (uint32_t)min(n0 + r, p.N - 1) * (uint32_t)p.K + (((lane & 7) ^ swizzle(r)) * 8);
    }
#define IEFWD_ISSUE(kt, slot)                                                                           \
    do {                                                                                                \
        const int k0_ = (kt) * kBK;                                                                     \
        bf16_t *ring_ = ring0 + (slot) * STAGE;                                                         \
        _Pragma("unroll") for (int i = 0; i < A_PW; ++i)                                                \
            __builtin_amdgcn_global_load_lds((const void *)(p.a + a_src[i] + k0_),                      \
                                             (lds_ptr_t)(ring_ + (wave + 4 * i) * 512), 16, 0, 0);      \
        _Pragma("unroll") for (int i = 0; i < W_PW; ++i)                                                \
            __builtin_amdgcn_global_load_lds((const void *)(p.w + w_src[i] + k0_),                      \
                                             (lds_ptr_t)(ring_ + BM * kBK + (wave + 4 * i) * 512), 16,  \
                                             0, 0);                                                     \
    } while (0)

#pragma unroll
    for (int s = 0; s < S - 1; ++s)
        if (s < n_mine) IEFWD_ISSUE(kt_first + s * kt_stride, s);

    // fragment rows: lane % 16 of each 16-row block; 16-byte chunk 4 ks + lane / 16
    const int ra = wm * TM + (lane & 15), rw = wn * TN + (lane & 15);
    for (int it = 0; it < n_steps; ++it) {
        // this wave's copies of its tile `it` are done once at most the later
        // tiles' copies are outstanding; the barrier then publishes every wave's
        // copies and guarantees the slot reused below is no longer being read
        if (it + S - 2 < n_mine)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm((S - 2) * LPW));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");   // keep LDS accesses on their side of the barrier
        if (it + S - 1 < n_mine) IEFWD_ISSUE(kt_first + (it + S - 1) * kt_stride, (it + S - 1) % S);
        if (it >= n_mine) continue;
        const bf16_t *ring = ring0 + (it % S) * STAGE;
#pragma unroll
        for (int ks = 0; ks < kBK / 32; ++ks) {
            const int c = ks * 4 + (lane >> 4);
            bf16x8 af[FM], wf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int r = ra + i * 16;
                af[i] = *reinterpret_cast<const bf16x8 *>(ring + r * kBK + ((c ^ swizzle(r)) * 8));
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int r = rw + j * 16;
                wf[j] = *reinterpret_cast<const bf16x8 *>(ring + BM * kBK + r * kBK + ((c ^ swizzle(r)) * 8));
            }
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], af[i], acc[j][i], 0, 0, 0);
        }
    }
#undef IEFWD_ISSUE
}

// Epilogue operands that do not depend on the product (bias, residual rows,
// LayerNorm statistics and affine) are loaded into registers before the main
// loop, so their latency hides behind the MFMAs instead of stalling the tail.
// The residual rows are prefetched only by 4-wave workgroups with small wave
// tiles (<= 6 blocks); larger tiles, and the 8-wave split workgroups (whose
// register budget is shared by both groups), would trade occupancy for it and
// load them in the epilogue instead.
template <int BM, int BN, Epi EPI, bool SPLIT = false>
struct EpiInputs {
    static constexpr int FM = BM / 32, FN = BN / 32;
    static constexpr bool kZ = (EPI == Epi::BiasResidF32 || EPI == Epi::BiasLnResidF32) && FN * FM <= 6 && !SPLIT;
    u32x2 bias[FN];
    f32x4 z[kZ ? FN : 1][kZ ? FM : 1];
    f32x2 stats[EPI == Epi::BiasLnResidF32 ? FM : 1];
    f32x4 gamma[EPI == Epi::BiasLnResidF32 ? FN : 1], beta[EPI == Epi::BiasLnResidF32 ? FN : 1];
};

template <int BM, int BN, Epi EPI, bool SPLIT>
__device__ inline void epilogue_prefetch(const GemmParams &p, EpiInputs<BM, BN, EPI, SPLIT> &in, int wave,
                                         int lane, int m0, int n0) {
    constexpr int TM = BM / 2, TN = BN / 2, FM = TM / 16, FN = TN / 16;
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int f = min(n0 + wn * TN + j * 16 + (lane >> 4) * 4, p.N - 4);
        in.bias[j] = *reinterpret_cast<const u32x2 *>(p.bias + f);
        if constexpr (EPI == Epi::BiasLnResidF32) {
            in.gamma[j] = *reinterpret_cast<const f32x4 *>(p.ln.gamma + f);
            in.beta[j] = *reinterpret_cast<const f32x4 *>(p.ln.beta + f);
        }
        if constexpr (EpiInputs<BM, BN, EPI, SPLIT>::kZ) {
            const float *src = EPI == Epi::BiasResidF32 ? p.resid : p.ln.z;
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int t = min(m0 + wm * TM + i * 16 + (lane & 15), p.M - 1);   // clamped: never stored
                in.z[j][i] = *reinterpret_cast<const f32x4 *>(src + (size_t)t * p.N + f);
            }
        }
    }
    if constexpr (EPI == Epi::BiasLnResidF32) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int t = min(m0 + wm * TM + i * 16 + (lane & 15), p.M - 1);
            in.stats[i] = *reinterpret_cast<const f32x2 *>(p.ln.stats + 2 * (size_t)t);
        }
    }
}

// Epilogue of one wave: lane owns features f..f+3 of token t in every block.
template <int BM, int BN, Epi EPI, bool SPLIT>
__device__ inline void epilogue(const GemmParams &p, const f32x4 (&acc)[BN / 32][BM / 32],
                                const EpiInputs<BM, BN, EPI, SPLIT> &in, int wave, int lane, int m0, int n0) {
    constexpr int TM = BM / 2, TN = BN / 2, FM = TM / 16, FN = TN / 16;
    const int wm = wave >> 1, wn = wave & 1;
    int tok[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) tok[i] = m0 + wm * TM + i * 16 + (lane & 15);
    int tok_b[FM], tok_s[FM];   // (sequence, position) of each token, for the head scatter
    if constexpr (EPI == Epi::Qkv) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            tok_b[i] = tok[i] / p.qkv.seq;
            tok_s[i] = tok[i] - tok_b[i] * p.qkv.seq;
        }
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int f = n0 + wn * TN + j * 16 + (lane >> 4) * 4;
        if (f >= p.N) continue;
        const u32x2 braw = in.bias[j];
        const float b0 = __uint_as_float(braw[0] << 16), b1 = __uint_as_float(braw[0] & 0xffff0000u);
        const float b2 = __uint_as_float(braw[1] << 16), b3 = __uint_as_float(braw[1] & 0xffff0000u);
        int which = 0, head = 0, jj = 0;   // head scatter: Q/K/V block, head, column within head
        if constexpr (EPI == Epi::Qkv) {
            which = f / p.qkv.d_model;
            const int within = f - which * p.qkv.d_model;
            head = within / p.qkv.head_dim;
            jj = within - head * p.qkv.head_dim;
        }
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int t = tok[i];
            if (t >= p.M) continue;
            float v0 = acc[j][i][0] + b0, v1 = acc[j][i][1] + b1;
            float v2 = acc[j][i][2] + b2, v3 = acc[j][i][3] + b3;
            if constexpr (EPI == Epi::BiasBf16 || EPI == Epi::BiasGeluBf16) {
                if constexpr (EPI == Epi::BiasGeluBf16) {
                    v0 = gelu(v0); v1 = gelu(v1); v2 = gelu(v2); v3 = gelu(v3);
                }
                bf16_t *o = static_cast<bf16_t *>(p.out) + (size_t)t * p.N + f;
                *reinterpret_cast<u32x2 *>(o) = u32x2{pack2(v0, v1), pack2(v2, v3)};
            } else if constexpr (EPI == Epi::BiasResidF32) {
                f32x4 r;
                if constexpr (EpiInputs<BM, BN, EPI, SPLIT>::kZ) r = in.z[j][i];
                else r = *reinterpret_cast<const f32x4 *>(p.resid + (size_t)t * p.N + f);
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) =
                    f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
            } else if constexpr (EPI == Epi::BiasLnResidF32) {
                // residual = LN(z) rebuilt with the LayerNorm kernel's expression
                f32x4 z;
                if constexpr (EpiInputs<BM, BN, EPI, SPLIT>::kZ) z = in.z[j][i];
                else z = *reinterpret_cast<const f32x4 *>(p.ln.z + (size_t)t * p.N + f);
                const float mean = in.stats[i][0], rstd = in.stats[i][1];
                f32x4 r;
#pragma unroll
                for (int e = 0; e < 4; ++e) r[e] = __builtin_fmaf(in.gamma[j][e], (z[e] - mean) * rstd, in.beta[j][e]);
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) =
                    f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
            } else {   // Epi::Qkv
                const QkvDst &d = p.qkv;
                const size_t bh = (size_t)tok_b[i] * d.n_heads + head;
                const int sp = tok_s[i];
                if (which < 2) {
                    bf16_t *o = (which == 0 ? d.q : d.k) + (bh * d.seq + sp) * d.head_dim + jj;
                    *reinterpret_cast<u32x2 *>(o) = u32x2{pack2(v0, v1), pack2(v2, v3)};
                } else {
                    bf16_t *o = d.vt + (bh * d.head_dim + jj) * d.seq_pad + sp;
                    o[0] = f32_to_bf16(v0);
                    o[d.seq_pad] = f32_to_bf16(v1);
                    o[2 * d.seq_pad] = f32_to_bf16(v2);
                    o[3 * d.seq_pad] = f32_to_bf16(v3);
                }
            }
        }
    }
}

// Sequential K order: 4 waves, one ring, K tiles 0, 1, 2, ... into one accumulator.
template <int BM, int BN, int S, Epi EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p) {
    __shared__ __attribute__((aligned(1024))) bf16_t lds[S * (BM + BN) * kBK];
    int tm, tn;
    grouped_tile(xcd_contiguous(blockIdx.x, gridDim.x), p.tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    f32x4 acc[BN / 32][BM / 32];
#pragma unroll
    for (int j = 0; j < BN / 32; ++j)
#pragma unroll
        for (int i = 0; i < BM / 32; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    EpiInputs<BM, BN, EPI, false> in;
    epilogue_prefetch<BM, BN, EPI, false>(p, in, wave, lane, m0, n0);
    const int kt_count = p.K / kBK;
    main_loop<BM, BN, S>(p, lds, wave, lane, m0, n0, 0, 1, kt_count, kt_count, acc);
    epilogue<BM, BN, EPI, false>(p, acc, in, wave, lane, m0, n0);
}

// Split K order: 8 waves in two 4-wave groups over the same output tile; group g
// accumulates the K tiles kt = g (mod 2) through its own ring, then group 1
// hands its partial sums to group 0 through LDS and group 0 adds them
// (even-tile sum + odd-tile sum, always in that order) and runs the epilogue.
// Two waves per SIMD even when there are only as many tiles as CUs.
template <int BM, int BN, int S, Epi EPI>
__global__ __launch_bounds__(2 * kThreads) void gemm_split_kernel(GemmParams p) {
    constexpr int FN = BN / 32, FM = BM / 32;
    __shared__ __attribute__((aligned(1024))) bf16_t lds[2 * S * (BM + BN) * kBK];
    static_assert(FN * FM * 4 * kThreads * 4 <= 2 * S * (BM + BN) * kBK * 2, "hand-off space");
    int tm, tn;
    grouped_tile(xcd_contiguous(blockIdx.x, gridDim.x), p.tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int lane = threadIdx.x & 63, grp = threadIdx.x >> 8, wave = (threadIdx.x >> 6) & 3;
    f32x4 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    EpiInputs<BM, BN, EPI, true> in;
    if (grp == 0) epilogue_prefetch<BM, BN, EPI, true>(p, in, wave, lane, m0, n0);
    const int kt_count = p.K / kBK;
    const int n_mine = (kt_count - grp + 1) / 2;
    main_loop<BM, BN, S>(p, lds + grp * S * (BM + BN) * kBK, wave, lane, m0, n0, grp, 2, n_mine,
                         (kt_count + 1) / 2, acc);
    __syncthreads();   // both rings drained: reuse the LDS for the hand-off
    float *handoff = reinterpret_cast<float *>(lds) + (wave * 64 + lane) * (FN * FM * 4);
    if (grp == 1) {
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int i = 0; i < FM; ++i) *reinterpret_cast<f32x4 *>(handoff + (j * FM + i) * 4) = acc[j][i];
    }
    __syncthreads();
    if (grp == 1) return;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] += *reinterpret_cast<const f32x4 *>(handoff + (j * FM + i) * 4);
    epilogue<BM, BN, EPI, true>(p, acc, in, wave, lane, m0, n0);
}

struct TileChoice {
    int bm, bn, stages;
    bool split;
};

// K summation order from the weight shape (N, K) only: K >= 2048 uses the
// split (even/odd) order, shorter K the sequential order.  So a given weight
// matrix always sums each output in the same order, whatever M (the batch),
// the CU quota or the tile shape -- outputs stay bit-identical across them.
bool split_k_order(int /*N*/, int K) { return K >= 2048; }

// Tile shape and ring depth from (M, N, K) only -- never the current CU quota.
// Measured inside the forward pass on gfx950: 64 x 96 tiles with a 2-slot ring
// (up to four workgroups per CU) win up to ~1500 such tiles, 128 x 96 beyond;
// 128 x 128 / 64 x 128 serve widths that 96 does not divide.  The split order
// runs 8-wave workgroups.
TileChoice choose_tile(int M, int N, int K) {
    const long m64 = (M + 63) / 64;
    if (split_k_order(N, K)) {
        if (N % 96 == 0) return {64, 96, 2, true};
        if (N % 128 == 0 && m64 * (N / 128) < 512) return {64, 128, 2, true};
        return {128, 128, 2, true};
    }
    if (N % 96 == 0 && m64 * (N / 96) <= 1536) return {64, 96, 2, false};
    if (N % 96 == 0) return {128, 96, 2, false};
    if (N % 128 == 0) return m64 * (N / 128) < 512 ? TileChoice{64, 128, 2, false} : TileChoice{128, 128, 2, false};
    return {64, 64, 3, false};
}

template <int BM, int BN, int S, bool SPLIT>
hipError_t launch_tile(Epi epi, GemmParams &p, hipStream_t s) {
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = p.N / BN;
    const dim3 grid(p.tiles_m * p.tiles_n), block(SPLIT ? 2 * kThreads : kThreads);
#define IEFWD_K(E) (SPLIT ? gemm_split_kernel<BM, BN, S, E> : gemm_kernel<BM, BN, S, E>)
    switch (epi) {
    case Epi::BiasBf16: return launch_kernel(IEFWD_K(Epi::BiasBf16), grid, block, s, p);
    case Epi::BiasGeluBf16: return launch_kernel(IEFWD_K(Epi::BiasGeluBf16), grid, block, s, p);
    case Epi::BiasResidF32: return launch_kernel(IEFWD_K(Epi::BiasResidF32), grid, block, s, p);
    case Epi::Qkv: return launch_kernel(IEFWD_K(Epi::Qkv), grid, block, s, p);
    case Epi::BiasLnResidF32: return launch_kernel(IEFWD_K(Epi::BiasLnResidF32), grid, block, s, p);
    }
#undef IEFWD_K
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                       const float *resid, void *out, int M, int N, int K, const QkvDst *qkv,
                       hipStream_t stream, const LnResid *ln) {
    if (M <= 0) return hipSuccess;
    GemmParams p{};
    p.a = a; p.w = w; p.bias = bias; p.resid = resid; p.out = out;
    p.M = M; p.N = N; p.K = K;
    if (qkv) p.qkv = *qkv;
    if (ln) p.ln = *ln;
    const TileChoice t = choose_tile(M, N, K);
    if (t.split) {
        if (t.bm == 64 && t.bn == 96) return launch_tile<64, 96, 2, true>(epi, p, stream);
        if (t.bm == 64 && t.bn == 128) return launch_tile<64, 128, 2, true>(epi, p, stream);
        return launch_tile<128, 128, 2, true>(epi, p, stream);
    }
    if (t.bm == 64 && t.bn == 96) return launch_tile<64, 96, 2, false>(epi, p, stream);
    if (t.bm == 64 && t.bn == 128) return launch_tile<64, 128, 2, false>(epi, p, stream);
    if (t.bm == 128 && t.bn == 128) return launch_tile<128, 128, 2, false>(epi, p, stream);
    if (t.bm == 128 && t.bn == 96) return launch_tile<128, 96, 2, false>(epi, p, stream);
    return launch_tile<64, 64, 3, false>(epi, p, stream);
}

}  // namespace iefwd
