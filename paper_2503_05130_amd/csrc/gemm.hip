// bf16 MFMA GEMM with fused epilogues for gfx950 (CDNA4).
//
// out[t, f] = epilogue( sum_k A[t, k] * W[f, k] + bias[f] )
//   A: activations, bf16 [M, K] row-major (tokens x features-in)
//   W: weights stored output-major, bf16 [N, K] row-major
//
// Both operands are K-contiguous, so every MFMA operand fragment is one 16-byte
// LDS read.  The kernel computes C^T blocks (features x tokens) with
// v_mfma_f32_16x16x32_bf16: the W fragment is the MFMA "A" operand and the
// activation fragment the "B" operand, so each lane ends up owning 4
// consecutive output features of one token and stores them with one vector
// store.
//
// Determinism and batch invariance: every tile configuration uses the same MFMA
// instruction and walks K in the same order (64-wide K tiles, two 32-wide MFMA
// steps each), so out[t, f] depends only on row t of A and row f of W -- never
// on the tile shape, the grid, the CU mask or the other rows in the batch.
// No atomics, no split-K.
#include "kernels.h"

#include <algorithm>

namespace iefwd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBK = 64;               // K tile (bf16 elements) = 128 bytes per row
constexpr int kLdsStride = kBK + 8;   // 144-byte LDS rows: 16 consecutive rows hit 16
                                      // distinct 16-byte bank groups for ds_read_b128
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

// GELU with the exact erf form.
__device__ inline float gelu(float u) { return 0.5f * u * (1.0f + erff(u * 0.7071067811865476f)); }

template <int BM, int BN, Epi EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmParams p) {
    constexpr int TM = BM / 2, TN = BN / 2;          // per-wave tile (tokens x features)
    constexpr int FM = TM / 16, FN = TN / 16;        // 16x16 MFMA blocks per wave
    constexpr int A_CH = BM * (kBK / 8) / kThreads;  // 16-byte chunks per thread
    constexpr int B_CH = BN * (kBK / 8) / kThreads;
    static_assert(BM * (kBK / 8) % kThreads == 0 && BN * (kBK / 8) % kThreads == 0, "tile");
    static_assert(TM % 16 == 0 && TN % 16 == 0, "wave tile");

    __shared__ __attribute__((aligned(16))) bf16_t lds[2 * (BM + BN) * kLdsStride];

    int tm, tn;
    grouped_tile(xcd_contiguous(blockIdx.x, gridDim.x), p.tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // This thread's global->LDS chunks: rows (tid / 8) + 32 i, 16-byte column
    // (tid % 8).  Rows past M / N are clamped to the last valid row (their
    // results are never stored).
    const int ld_row = tid >> 3, ld_col = (tid & 7) * 8;
    uint32_t a_off[A_CH], w_off[B_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i)
        a_off[i] = (uint32_t)min(m0 + ld_row + 32 * i, p.M - 1) * (uint32_t)p.K + ld_col;
#pragma unroll
    for (int i = 0; i < B_CH; ++i)
        w_off[i] = (uint32_t)min(n0 + ld_row + 32 * i, p.N - 1) * (uint32_t)p.K + ld_col;
    const int st_off = ld_row * kLdsStride + ld_col;

    u32x4 ra[A_CH], rw[B_CH];
#define IEFWD_GLOAD(k0)                                                                   \
    do {                                                                                  \
        _Pragma("unroll") for (int i = 0; i < A_CH; ++i)                                  \
            ra[i] = *reinterpret_cast<const u32x4 *>(p.a + a_off[i] + (k0));              \
        _Pragma("unroll") for (int i = 0; i < B_CH; ++i)                                  \
            rw[i] = *reinterpret_cast<const u32x4 *>(p.w + w_off[i] + (k0));              \
    } while (0)
#define IEFWD_LSTORE(buf)                                                                 \
    do {                                                                                  \
        bf16_t *base_ = lds + (buf) * (BM + BN) * kLdsStride + st_off;                    \
        _Pragma("unroll") for (int i = 0; i < A_CH; ++i)                                  \
            *reinterpret_cast<u32x4 *>(base_ + 32 * i * kLdsStride) = ra[i];              \
        _Pragma("unroll") for (int i = 0; i < B_CH; ++i)                                  \
            *reinterpret_cast<u32x4 *>(base_ + (BM + 32 * i) * kLdsStride) = rw[i];       \
    } while (0)

    f32x4 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // fragment read offsets: row = lane % 16 of each 16-row block, k = 8 * (lane / 16)
    const int a_frag = (wm * TM + (lane & 15)) * kLdsStride + (lane >> 4) * 8;
    const int w_frag = BM * kLdsStride + (wn * TN + (lane & 15)) * kLdsStride + (lane >> 4) * 8;

    const int kt_count = p.K / kBK;
    IEFWD_GLOAD(0);
    IEFWD_LSTORE(0);
    __syncthreads();
    for (int kt = 0; kt < kt_count; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < kt_count) IEFWD_GLOAD((kt + 1) * kBK);   // in flight during the MFMAs
        const bf16_t *base = lds + buf * (BM + BN) * kLdsStride;
#pragma unroll
        for (int ks = 0; ks < kBK / 32; ++ks) {
            bf16x8 af[FM], wf[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                af[i] = *reinterpret_cast<const bf16x8 *>(base + a_frag + i * 16 * kLdsStride + ks * 32);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                wf[j] = *reinterpret_cast<const bf16x8 *>(base + w_frag + j * 16 * kLdsStride + ks * 32);
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], af[i], acc[j][i], 0, 0, 0);
        }
        if (kt + 1 < kt_count) IEFWD_LSTORE(buf ^ 1);
        __syncthreads();
    }
#undef IEFWD_GLOAD
#undef IEFWD_LSTORE

    // Epilogue: lane owns features f..f+3 of token t in every block.
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int f = n0 + wn * TN + j * 16 + (lane >> 4) * 4;
        if (f >= p.N) continue;
        const u32x2 braw = *reinterpret_cast<const u32x2 *>(p.bias + f);
        const float b0 = __uint_as_float(braw.x << 16), b1 = __uint_as_float(braw.x & 0xffff0000u);
        const float b2 = __uint_as_float(braw.y << 16), b3 = __uint_as_float(braw.y & 0xffff0000u);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int t = m0 + wm * TM + i * 16 + (lane & 15);
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
                const size_t off = (size_t)t * p.N + f;
                const f32x4 r = *reinterpret_cast<const f32x4 *>(p.resid + off);
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + off) =
                    f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
            } else {   // Epi::Qkv
                const QkvDst &d = p.qkv;
                const int which = f / d.d_model;               // 0 Q, 1 K, 2 V
                const int within = f - which * d.d_model;
                const int h = within / d.head_dim, jj = within - h * d.head_dim;
                const int b = t / d.seq, s = t - b * d.seq;
                const size_t bh = (size_t)b * d.n_heads + h;
                if (which < 2) {
                    bf16_t *o = (which == 0 ? d.q : d.k) + (bh * d.seq + s) * d.head_dim + jj;
                    *reinterpret_cast<u32x2 *>(o) = u32x2{pack2(v0, v1), pack2(v2, v3)};
                } else {
                    bf16_t *o = d.vt + (bh * d.head_dim + jj) * d.seq_pad + s;
                    o[0] = f32_to_bf16(v0);
                    o[d.seq_pad] = f32_to_bf16(v1);
                    o[2 * d.seq_pad] = f32_to_bf16(v2);
                    o[3 * d.seq_pad] = f32_to_bf16(v3);
                }
            }
        }
    }
}

struct TileChoice {
    int bm, bn;
};

// Tile shape from (M, N) only -- a fixed cost model of whole-chip rounds of 256
// workgroups, never the current CU quota.  Smaller tiles pay a per-output
// overhead factor for their lower operand reuse.
TileChoice choose_tile(int M, int N) {
    struct Cand { int bm, bn; double overhead; };
    static const Cand cands[] = {{128, 128, 1.00}, {128, 96, 1.05}, {128, 64, 1.15}, {64, 64, 1.40}};
    TileChoice best{128, 128};
    double best_cost = 1e300;
    for (const Cand &c : cands) {
        if (N % c.bn != 0) continue;
        const long tiles = (long)((M + c.bm - 1) / c.bm) * (N / c.bn);
        const long rounds = (tiles + 255) / 256;
        const double cost = (double)rounds * c.bm * c.bn * c.overhead;
        if (cost < best_cost) { best_cost = cost; best = {c.bm, c.bn}; }
    }
    return best;
}

template <int BM, int BN>
hipError_t launch_tile(Epi epi, GemmParams &p, hipStream_t s) {
    p.tiles_m = (p.M + BM - 1) / BM;
    p.tiles_n = p.N / BN;
    const dim3 grid(p.tiles_m * p.tiles_n), block(kThreads);
    switch (epi) {
    case Epi::BiasBf16: hipLaunchKernelGGL((gemm_kernel<BM, BN, Epi::BiasBf16>), grid, block, 0, s, p); break;
    case Epi::BiasGeluBf16: hipLaunchKernelGGL((gemm_kernel<BM, BN, Epi::BiasGeluBf16>), grid, block, 0, s, p); break;
    case Epi::BiasResidF32: hipLaunchKernelGGL((gemm_kernel<BM, BN, Epi::BiasResidF32>), grid, block, 0, s, p); break;
    case Epi::Qkv: hipLaunchKernelGGL((gemm_kernel<BM, BN, Epi::Qkv>), grid, block, 0, s, p); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                       const float *resid, void *out, int M, int N, int K, const QkvDst *qkv,
                       hipStream_t stream) {
    if (M <= 0) return hipSuccess;
    GemmParams p{};
    p.a = a; p.w = w; p.bias = bias; p.resid = resid; p.out = out;
    p.M = M; p.N = N; p.K = K;
    if (qkv) p.qkv = *qkv;
    const TileChoice t = choose_tile(M, N);
    if (t.bm == 128 && t.bn == 128) return launch_tile<128, 128>(epi, p, stream);
    if (t.bm == 128 && t.bn == 96) return launch_tile<128, 96>(epi, p, stream);
    if (t.bm == 128 && t.bn == 64) return launch_tile<128, 64>(epi, p, stream);
    return launch_tile<64, 64>(epi, p, stream);
}

}  // namespace iefwd
