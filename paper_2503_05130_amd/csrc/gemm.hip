// bf16 MFMA GEMM with fused epilogues for gfx950 (CDNA4).
//
// out[t, f] = epilogue( sum_k A[t, k] * W[f, k] + bias[f] )
//   A: activations, bf16 [M, K] row-major (tokens x features-in)
//   W: weights stored output-major, bf16 [N, K] row-major
//
// Data movement.  K is walked in BK-wide tiles (64, or 32 for a deeper ring).
// Each tile of A and W is copied from global memory straight into LDS with
// global_load_lds_dwordx4 (gfx950's 16-byte global->LDS DMA: no VGPR
// staging) into an S-slot ring shared by the workgroup's wave groups; a
// tile's 1 KB copies are spread over all waves.  LDS rows hold BK elements
// with the 16-byte chunks XOR-swizzled per row, so that the 16 rows read by
// one ds_read_b128 fragment load fall in distinct banks; the swizzle is
// applied on the source side (lane i of a DMA fetches the global chunk that
// belongs at its fixed LDS slot).  Each wave waits for its own copies of the
// tiles it is about to read (s_waitcnt vmcnt), then a workgroup barrier makes
// every wave's copies visible and frees the slots the next copies overwrite.
// The MFMAs of each 32-deep half tile are issued before the LDS reads of the
// next half, so fragment reads overlap the matrix unit's work.
//
// Math.  v_mfma_f32_16x16x32_bf16 on C^T blocks (features x tokens): the W
// fragment is the MFMA "A" operand, the activation fragment the "B" operand,
// so each lane ends up owning 4 consecutive output features of one token and
// stores them with one vector store.
//
// Determinism and batch invariance: every configuration uses the same MFMA
// instruction; the K summation order (32-wide K chunks in sequence, or the
// workgroup-internal even/odd split of 64-wide tiles for long K) is a function
// of the weight shape (N, K) alone.  So out[t, f] depends only on row t of A
// and row f of W -- never on the tile shape, the ring depth, the grid, the CU
// mask or the other rows in the batch.  No atomics, no cross-workgroup split-K.
#include "gelu.h"
#include "gemm.h"

#include <algorithm>

namespace iefwd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void *lds_ptr_t;

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
    LnIn lnin;
    const bf16_t *aux;   // Epi::GeluBwdBf16: the GELU's input [M, N]
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

template <int CTRL>
__device__ inline float dpp_move(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}

// Sum over the wave's 64 lanes, the same value in every lane, in a fixed
// order: lane pairs and pairs of pairs within each quad (DPP quad permutes
// [1,0,3,2] and [2,3,0,1]), quads within each half row (row_half_mirror),
// halves within each row of 16 (row_mirror), then the four row sums as
// (r0 + r1) + (r2 + r3).  Each partner exchange adds the same two values in
// both lanes, so every lane of a group holds bitwise the same sum.
__device__ inline float wave_sum(float v) {
    v += dpp_move<0xB1>(v);
    v += dpp_move<0x4E>(v);
    v += dpp_move<0x141>(v);
    v += dpp_move<0x140>(v);
    const int b = __builtin_bit_cast(int, v);
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48));
    return (r0 + r1) + (r2 + r3);
}

// 16-byte chunk position of logical chunk 0 in LDS row r of a BK-wide K tile
// (row r holds its chunk c at position c ^ swizzle<BK>(r)), chosen so that the
// 16 rows one ds_read_b128 fragment load reads fall in distinct banks:
//  - 128-byte rows (BK = 64): consecutive rows alternate between the two
//    128-byte halves of a 256-byte bank line, and within each parity the 8
//    rows of a 16-row fragment get 8 distinct positions;
//  - 64-byte rows (BK = 32): rows r, r + 4, r + 8, r + 12 share a bank offset
//    and get the 4 distinct positions.
template <int BK>
__device__ inline int swizzle(int r) {
    if constexpr (BK == 64) return ((r >> 1) & 7) ^ ((r & 1) << 2);
    else return (r >> 2) & 3;
}

// One global->LDS copy of 16 bytes per lane (1 KB per wave) to the
// wave-uniform LDS byte address `lds`.  Issued through inline asm: the
// compiler's wait-count model treats these copies as LDS traffic that may
// complete out of order with LDS reads, and would then drain every
// outstanding LDS read before each use of any of them; the main loop orders
// the copies itself (s_waitcnt vmcnt before each barrier).  The M0 write
// needs one wait state before the copy reads it.
__device__ inline void dma16(const void *src, uint32_t lds) {
    uint32_t m0;   // the asm writes M0; naming it as an output tells the compiler so
    asm volatile("s_mov_b32 %0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 : "={m0}"(m0)
                 : "v"(src), "s"(lds)
                 : "memory");
    (void)m0;
}

// s_waitcnt immediate: wait until at most vm vector-memory and lgkm LDS
// operations of this wave are outstanding (expcnt left unconstrained).
constexpr int waitcnt_imm(int vm, int lgkm) { return (vm & 15) | (7 << 4) | ((lgkm & 15) << 8) | ((vm >> 4) << 14); }

// Tile configuration: BM x BN output tile; G wave groups of WGM x WGN waves;
// one S-slot LDS ring of BK-wide K tiles (BK = 32 or 64) shared by the groups.
// The MFMA sums 32 K at a time; G is the K order: G = 1 adds the 32-wide K
// chunks in sequence (the same order for either BK), G = 2 (BK = 64 only) has
// group g sum the 64-wide K tiles with index = g (mod 2) in sequence, then
// adds the two partial sums.
template <int BM_, int BN_, int WGM_, int WGN_, int G_, int S_, int BK_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, G = G_, S = S_, BK = BK_;
    static constexpr int NWG = WGM * WGN;                      // waves per group
    static constexpr int NW = G * NWG, NT = 64 * NW;           // waves / threads per workgroup
    static constexpr int TM = BM / WGM, TN = BN / WGN;         // per-wave tile (tokens x features)
    static constexpr int FM = TM / 16, FN = TN / 16;           // 16 x 16 MFMA blocks per wave
    static constexpr int H = BK / 32;                          // 32-deep MFMA steps per K tile
    static constexpr int CPR = BK / 8;                         // 16-byte chunks per LDS row
    static constexpr int RPG = 64 / CPR;                       // rows per 1 KB DMA (64 lanes x 16 B)
    static constexpr int STAGE = (BM + BN) * BK;               // bf16 elements per ring slot
    static constexpr int DG = (BM + BN) / RPG;                 // 1 KB DMA groups per slot
    static constexpr int DPW = (DG + NW - 1) / NW;             // DMA groups per wave per slot (at most)
    // waves per SIMD the register budget is sized for: as many workgroups as
    // the LDS ring allows share a CU (160 KB), at most 4 waves per SIMD
    static constexpr int WG_CU = 163840 / (S * STAGE * 2);
    static constexpr int WPE = WG_CU * NW / 4 >= 4 ? 4 : WG_CU * NW / 4 < 1 ? 1 : WG_CU * NW / 4;
    static_assert(TM % 16 == 0 && TN % 16 == 0 && BM % RPG == 0 && BN % RPG == 0, "tile");
    static_assert(BK == 32 || BK == 64, "K tile");
    static_assert(G == 1 || (G == 2 && BK == 64), "K order");
    static_assert(S >= 2 * G && (S - 1) * DPW <= 63, "ring depth (vmcnt holds 6 bits)");
};

// Waits until at most `t` K tiles' worth of this wave's copies (`per` DMAs
// each) are still in flight: the copies of tiles issued after the ones about
// to be read.  t in [0, S - 1]; the s_waitcnt immediate must be a constant,
// hence the recursion over the possible counts.
template <class C, int c = C::S - 1>
__device__ inline void wait_tiles(int t, int per) {
    if constexpr (c == 0) {
        __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));
    } else {
        if (t >= c) {
            if constexpr (C::DPW > 1) {
                if (per != C::DPW) {
                    __builtin_amdgcn_s_waitcnt(waitcnt_imm(c * (C::DPW - 1), 15));
                    return;
                }
            }
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(c * C::DPW, 15));
            return;
        }
        wait_tiles<C, c - 1>(t, per);
    }
}

// The main loop over the K tiles through the shared ring.  Tile t lives in
// slot t % S; step j has group g multiply tile jG + g, 32 K at a time (H =
// BK / 32 halves per tile).  Each half's MFMAs are issued before the LDS
// reads of the next half, so those reads run while the matrix unit works
// through the MFMAs just queued; the barrier sits between a step's last
// reads and the next step's first ones:
//
//   MFMAs of half h                   (fragments read before)
//   h < H - 1: read half h + 1 of my tile
//   h = H - 1: wait for my copies of the next step's tiles and my LDS reads;
//              barrier (next tiles visible to all; no wave reads this
//              step's slots any more); refill this step's slots with tiles
//              jG + S .. jG + S + G - 1; read half 0 of my next tile
//
// so S - G tiles are in flight behind the ones being read.  Each tile's 1 KB
// copies are spread over all the workgroup's waves.
template <class C>
__device__ inline void main_loop(const GemmParams &p, bf16_t *ring0, int wave, int lane, int m0, int n0,
                                 f32x4 (&acc)[C::FN][C::FM]) {
    constexpr int NW = C::NW, DPW = C::DPW, DG = C::DG, S = C::S, G = C::G, FM = C::FM, FN = C::FN;
    constexpr int BK = C::BK, H = C::H, CPR = C::CPR, RPG = C::RPG;
    const int grp = wave / C::NWG, gw = wave % C::NWG;
    const int wm = gw % C::WGM, wn = gw / C::WGM;

    // DMA sources of this lane: DMA i of this wave copies the RPG-row group
    // d = wave + NW i of a slot (A rows first, then W rows); lane l fills row
    // RPG d + l / CPR of the slot at chunk position l % CPR.  Rows past M are
    // clamped to the last valid row (never stored); N is a multiple of BN.
    uint32_t src[DPW];
    const bf16_t *base[DPW];
    int per = 0;   // DMAs this wave issues per tile
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
        const int d = min(wave + NW * i, DG - 1);
        per += wave + NW * i < DG;
        if (d < C::BM / RPG) {
            const int r = RPG * d + lane / CPR;
            src[i] = (uint32_t)min(m0 + r, p.M - 1) * (uint32_t)p.K + (((lane % CPR) ^ swizzle<BK>(r)) * 8);
            base[i] = p.a;
        } else {
            const int r = RPG * (d - C::BM / RPG) + lane / CPR;
            src[i] = (uint32_t)(n0 + r) * (uint32_t)p.K + (((lane % CPR) ^ swizzle<BK>(r)) * 8);
            base[i] = p.w;
        }
    }
    const int n_kt = p.K / BK;
    auto issue = [&](int t) {   // copies of K tile t into slot t % S
        const int k0 = t * BK;
        bf16_t *ring = ring0 + (t % S) * C::STAGE;
#pragma unroll
        for (int i = 0; i < DPW; ++i)
            if (wave + NW * i < DG)
                dma16(base[i] + src[i] + k0, (uint32_t)(size_t)(lds_ptr_t)(ring + (wave + NW * i) * 512));
    };
    // fragment rows: lane % 16 of each 16-row block; 16-byte chunk 4 half + lane / 16
    const int ra = wm * C::TM + (lane & 15), rw = wn * C::TN + (lane & 15);
    auto read = [&](bf16x8 (&af)[FM], bf16x8 (&wf)[FN], int t, int half) {
        const bf16_t *ring = ring0 + (t % S) * C::STAGE;
        const int c = half * 4 + (lane >> 4);
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int r = ra + i * 16;
            af[i] = *reinterpret_cast<const bf16x8 *>(ring + r * BK + ((c ^ swizzle<BK>(r)) * 8));
        }
#pragma unroll
        for (int jj = 0; jj < FN; ++jj) {
            const int r = rw + jj * 16;
            wf[jj] = *reinterpret_cast<const bf16x8 *>(ring + C::BM * BK + r * BK + ((c ^ swizzle<BK>(r)) * 8));
        }
    };
    auto mfma = [&](const bf16x8 (&af)[FM], const bf16x8 (&wf)[FN]) {
#pragma unroll
        for (int jj = 0; jj < FN; ++jj)
#pragma unroll
            for (int i = 0; i < FM; ++i)
                acc[jj][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[jj], af[i], acc[jj][i], 0, 0, 0);
    };

#pragma unroll
    for (int t = 0; t < S; ++t)
        if (t < n_kt) issue(t);
    bf16x8 a0[FM], w0[FN], a1[FM], w1[FN];
    wait_tiles<C>(min(n_kt, S) - min(n_kt, G), per);   // the first step's tiles have landed
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");   // keep LDS accesses on their side of the barrier
    if (grp < n_kt) read(a0, w0, grp, 0);
    const int n_steps = (n_kt + G - 1) / G, n_q = n_steps * H;
    // half-step q: step q / H, half q % H of this group's tile
    auto half = [&](bf16x8 (&ca)[FM], bf16x8 (&cw)[FN], bf16x8 (&na)[FM], bf16x8 (&nw)[FN], int q) {
        const int j = q / H, h = q % H, t = j * G + grp;
        if (t < n_kt) mfma(ca, cw);
        if (h + 1 < H) {
            if (t < n_kt) read(na, nw, t, h + 1);
        } else if (j + 1 < n_steps) {
            wait_tiles<C>(min(n_kt, j * G + S) - min(n_kt, (j + 2) * G), per);
            __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));   // my reads of this step's slots have returned
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
#pragma unroll
            for (int u = 0; u < G; ++u)
                if (j * G + S + u < n_kt) issue(j * G + S + u);
            if (t + G < n_kt) read(na, nw, t + G, 0);
        }
    };
    for (int q = 0; q < n_q; q += 2) {
        half(a0, w0, a1, w1, q);
        if (q + 1 < n_q) half(a1, w1, a0, w0, q + 1);
    }
}

// bf16 outputs (bias, bias + GELU, the QKV scatter) leave through LDS: each wave
// writes its finished values into an LDS copy of the output tile, then the
// whole workgroup stores it in 16-byte row segments.  Written straight from
// the MFMA layout, one store instruction would cover 16 rows x 32 bytes.
constexpr bool staged(Epi e) {
    return e == Epi::BiasBf16 || e == Epi::BiasGeluBf16 || e == Epi::Qkv || e == Epi::GeluBwdBf16;
}
constexpr bool has_bias(Epi e) { return e != Epi::F32 && e != Epi::GeluBwdBf16; }

// Epilogue operands that do not depend on the product (bias, residual rows,
// LayerNorm statistics and affine) are loaded into registers before the main
// loop, so their latency hides behind the MFMAs instead of stalling the tail.
// The residual rows are prefetched only by 4-wave workgroups with small wave
// tiles (<= 6 blocks); larger tiles, and the split workgroups (whose register
// budget is shared by both groups), would trade occupancy for it and load them
// in the epilogue instead.
template <class C, Epi EPI>
struct EpiInputs {
    static constexpr int FM = C::FM, FN = C::FN;
    static constexpr bool kZ =
        (EPI == Epi::BiasResidF32 || EPI == Epi::BiasLnResidF32) && FN * FM <= 6 && C::NW == 4 && C::G == 1;
    u32x2 bias[FN];
    f32x4 z[kZ ? FN : 1][kZ ? FM : 1];
    f32x2 stats[EPI == Epi::BiasLnResidF32 ? FM : 1];
    f32x4 gamma[EPI == Epi::BiasLnResidF32 ? FN : 1], beta[EPI == Epi::BiasLnResidF32 ? FN : 1];
};

template <class C, Epi EPI>
__device__ inline void epilogue_prefetch(const GemmParams &p, EpiInputs<C, EPI> &in, int wave, int lane,
                                         int m0, int n0) {
    const int wm = wave % C::WGM, wn = wave / C::WGM;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int f = n0 + wn * C::TN + j * 16 + (lane >> 4) * 4;
        if constexpr (has_bias(EPI)) in.bias[j] = *reinterpret_cast<const u32x2 *>(p.bias + f);
        else in.bias[j] = u32x2{0u, 0u};
        if constexpr (EPI == Epi::BiasLnResidF32) {
            in.gamma[j] = *reinterpret_cast<const f32x4 *>(p.ln.gamma + f);
            in.beta[j] = *reinterpret_cast<const f32x4 *>(p.ln.beta + f);
        }
        if constexpr (EpiInputs<C, EPI>::kZ) {
            const float *src = EPI == Epi::BiasResidF32 ? p.resid : p.ln.z;
#pragma unroll
            for (int i = 0; i < C::FM; ++i) {
                const int t = min(m0 + wm * C::TM + i * 16 + (lane & 15), p.M - 1);   // clamped: never stored
                in.z[j][i] = *reinterpret_cast<const f32x4 *>(src + (size_t)t * p.N + f);
            }
        }
    }
    if constexpr (EPI == Epi::BiasLnResidF32) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int t = min(m0 + wm * C::TM + i * 16 + (lane & 15), p.M - 1);
            in.stats[i] = *reinterpret_cast<const f32x2 *>(p.ln.stats + 2 * (size_t)t);
        }
    }
}

// Row strides (bf16) of the staged output tile: token-major for plain bf16
// outputs and Q/K, feature-major for V^T.  The 8-element pad keeps rows
// 16-byte aligned and spreads consecutive rows over the LDS banks.
template <class C> constexpr int kRowStride = C::BN + 8;
template <class C> constexpr int kColStride = C::BM + 8;

// Epilogue of one wave.  Lane owns features f..f+3 of token t in every block.
// fp32 outputs are stored directly (one 16-byte store per block); bf16 outputs
// go to the LDS tile `ctile` (token-major, or feature-major when `vt_tile`).
template <class C, Epi EPI>
__device__ inline void epilogue(const GemmParams &p, const f32x4 (&acc)[C::FN][C::FM],
                                const EpiInputs<C, EPI> &in, int wave, int lane, int m0, int n0,
                                bf16_t *ctile, bool vt_tile) {
    const int wm = wave % C::WGM, wn = wave / C::WGM;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
        const int fl = wn * C::TN + j * 16 + (lane >> 4) * 4;   // feature within the tile
        const int f = n0 + fl;
        const u32x2 braw = in.bias[j];
        const float b0 = __uint_as_float(braw[0] << 16), b1 = __uint_as_float(braw[0] & 0xffff0000u);
        const float b2 = __uint_as_float(braw[1] << 16), b3 = __uint_as_float(braw[1] & 0xffff0000u);
#pragma unroll
        for (int i = 0; i < C::FM; ++i) {
            const int tl = wm * C::TM + i * 16 + (lane & 15);   // token within the tile
            const int t = m0 + tl;
            float v0 = acc[j][i][0] + b0, v1 = acc[j][i][1] + b1;
            float v2 = acc[j][i][2] + b2, v3 = acc[j][i][3] + b3;
            if constexpr (staged(EPI)) {
                if constexpr (EPI == Epi::BiasGeluBf16) {
                    v0 = gelu(v0); v1 = gelu(v1); v2 = gelu(v2); v3 = gelu(v3);
                }
                if constexpr (EPI == Epi::GeluBwdBf16) {   // rows past M read row M - 1: never stored
                    const u32x2 g = *reinterpret_cast<const u32x2 *>(p.aux + (size_t)min(t, p.M - 1) * p.N + f);
                    v0 *= gelu_grad(__uint_as_float(g[0] << 16));
                    v1 *= gelu_grad(__uint_as_float(g[0] & 0xffff0000u));
                    v2 *= gelu_grad(__uint_as_float(g[1] << 16));
                    v3 *= gelu_grad(__uint_as_float(g[1] & 0xffff0000u));
                }
                if (EPI == Epi::Qkv && vt_tile) {
                    bf16_t *o = ctile + fl * kColStride<C> + tl;
                    o[0] = f32_to_bf16(v0);
                    o[kColStride<C>] = f32_to_bf16(v1);
                    o[2 * kColStride<C>] = f32_to_bf16(v2);
                    o[3 * kColStride<C>] = f32_to_bf16(v3);
                } else {
                    *reinterpret_cast<u32x2 *>(ctile + tl * kRowStride<C> + fl) = u32x2{pack2(v0, v1), pack2(v2, v3)};
                }
            } else if constexpr (EPI == Epi::F32) {
                if (t >= p.M) continue;
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) = f32x4{v0, v1, v2, v3};
            } else if constexpr (EPI == Epi::BiasResidF32) {
                if (t >= p.M) continue;
                f32x4 r;
                if constexpr (EpiInputs<C, EPI>::kZ) r = in.z[j][i];
                else r = *reinterpret_cast<const f32x4 *>(p.resid + (size_t)t * p.N + f);
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) =
                    f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
            } else {   // Epi::BiasLnResidF32: residual = LN(z) rebuilt with the LayerNorm kernel's expression
                if (t >= p.M) continue;
                f32x4 z;
                if constexpr (EpiInputs<C, EPI>::kZ) z = in.z[j][i];
                else z = *reinterpret_cast<const f32x4 *>(p.ln.z + (size_t)t * p.N + f);
                const float mean = in.stats[i][0], rstd = in.stats[i][1];
                f32x4 r;
#pragma unroll
                for (int e = 0; e < 4; ++e) r[e] = __builtin_fmaf(in.gamma[j][e], (z[e] - mean) * rstd, in.beta[j][e]);
                *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) =
                    f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
            }
        }
    }
}

// Store the staged bf16 tile.  Called by all `nt` threads of the workgroup
// after a barrier that follows every wave's epilogue().
template <class C, Epi EPI>
__device__ inline void store_tile(const GemmParams &p, const bf16_t *ctile, bool vt_tile, int tid, int nt, int m0,
                                  int n0) {
    if (EPI == Epi::Qkv && vt_tile) {
        // V^T [B, H, dh, vt_stride]: a segment is 8 consecutive tokens of one
        // (head, column) row, contiguous when seq and pos0 are multiples of 8
        const QkvDst &d = p.qkv;
        constexpr int TG = C::BM / 8;
        for (int sg = tid; sg < C::BN * TG; sg += nt) {
            const int fl = sg / TG, t0 = m0 + (sg % TG) * 8;
            if (t0 >= p.M) continue;
            const int within = n0 + fl - 2 * d.d_model, head = within / d.head_dim, jj = within - head * d.head_dim;
            const bf16_t *src = ctile + fl * kColStride<C> + (t0 - m0);
            if (d.seq % 8 == 0 && d.pos0 % 8 == 0) {
                const int b = t0 / d.seq, sp = d.pos0 + t0 - b * d.seq;
                bf16_t *o = d.vt + (((size_t)b * d.n_heads + head) * d.head_dim + jj) * d.vt_stride + sp;
                *reinterpret_cast<u32x4 *>(o) = *reinterpret_cast<const u32x4 *>(src);
            } else {
                for (int e = 0; e < 8 && t0 + e < p.M; ++e) {
                    const int t = t0 + e, b = t / d.seq, sp = d.pos0 + t - b * d.seq;
                    d.vt[(((size_t)b * d.n_heads + head) * d.head_dim + jj) * d.vt_stride + sp] = src[e];
                }
            }
        }
        return;
    }
    constexpr int SEGS = C::BN / 8;   // 16-byte segments per token row
    for (int sg = tid; sg < C::BM * SEGS; sg += nt) {
        const int r = sg / SEGS, c = sg - r * SEGS, t = m0 + r;
        if (t >= p.M) continue;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(ctile + r * kRowStride<C> + c * 8);
        const int f = n0 + c * 8;
        bf16_t *o;
        if constexpr (EPI == Epi::Qkv) {   // Q or K [B, H, S, dh]: 8 columns of one head
            const QkvDst &d = p.qkv;
            const int which = f / d.d_model, within = f - which * d.d_model;
            const int head = within / d.head_dim, jj = within - head * d.head_dim;
            const int b = t / d.seq, sp = t - b * d.seq;
            o = which == 0 ? d.q + (((size_t)b * d.n_heads + head) * d.seq + sp) * d.head_dim + jj
                           : d.k + (((size_t)b * d.n_heads + head) * d.k_rows + d.pos0 + sp) * d.head_dim + jj;
        } else {
            o = static_cast<bf16_t *>(p.out) + (size_t)t * p.N + f;
        }
        *reinterpret_cast<u32x4 *>(o) = v;
    }
}

// One output tile per workgroup.  With two wave groups (the even / odd K
// order) group 1 hands its partial sums to group 0 through LDS once the ring
// is drained, and group 0 adds them (even-tile sum + odd-tile sum, always in
// that order) and runs the epilogue.
template <class C, Epi EPI>
__global__ __launch_bounds__(C::NT) __attribute__((amdgpu_waves_per_eu(C::WPE))) void gemm_kernel(GemmParams p) {
    constexpr int FN = C::FN, FM = C::FM;
    __shared__ __attribute__((aligned(1024))) bf16_t lds[C::S * C::STAGE];
    static_assert(!staged(EPI) || (C::BM * kRowStride<C> <= C::S * C::STAGE &&
                                   C::BN * kColStride<C> <= C::S * C::STAGE), "staged tile fits in the ring");
    static_assert(C::G == 1 || FN * FM * 4 * C::NWG * 64 * 4 <= C::S * C::STAGE * 2, "hand-off space");
    int tm, tn;
    grouped_tile(xcd_contiguous(blockIdx.x, gridDim.x), p.tiles_m, p.tiles_n, tm, tn);
    const int m0 = tm * C::BM, n0 = tn * C::BN;
    // the wave index is uniform across the wave: held in a scalar register, so
    // that every branch on it (group, tile, copy counts) is a scalar branch
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wave / C::NWG, gw = wave % C::NWG;   // group, wave within the group
    f32x4 acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) acc[j][i] = f32x4{0.f, 0.f, 0.f, 0.f};
    EpiInputs<C, EPI> in;
    if (grp == 0) epilogue_prefetch<C, EPI>(p, in, gw, lane, m0, n0);
    main_loop<C>(p, lds, wave, lane, m0, n0, acc);
    __syncthreads();   // every wave is done reading the ring (and every copy has landed)
    if constexpr (C::G == 2) {
        float *handoff = reinterpret_cast<float *>(lds) + (gw * 64 + lane) * (FN * FM * 4);
        if (grp == 1) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) *reinterpret_cast<f32x4 *>(handoff + (j * FM + i) * 4) = acc[j][i];
        }
        __syncthreads();
        if (grp == 0) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i) acc[j][i] += *reinterpret_cast<const f32x4 *>(handoff + (j * FM + i) * 4);
        }
        if constexpr (staged(EPI)) __syncthreads();   // the hand-off is consumed before the tile overwrites it
    }
    const bool vt_tile = EPI == Epi::Qkv && n0 >= 2 * p.qkv.d_model;
    if (grp == 0) epilogue<C, EPI>(p, acc, in, gw, lane, m0, n0, lds, vt_tile);
    if constexpr (staged(EPI)) {
        __syncthreads();
        store_tile<C, EPI>(p, lds, vt_tile, threadIdx.x, C::NT, m0, n0);
    }
}

// Tile configurations.  8-wave workgroups for large tiles: two waves per SIMD
// and a 128-row tile halve the operand bytes each CU pulls through its L1 per
// MFMA compared with 64-row 4-wave tiles (the per-CU load path moves about
// 43 B/clk of global->LDS copies, which bounds small tiles below the MFMA rate).
//                BM   BN  WGM WGN G  S  BK
using CfgA = Cfg<128, 192, 2, 4, 1, 2, 64>;   // 8 waves, 64 x 48 per wave; 2 per CU
using CfgD = Cfg<128, 128, 2, 4, 1, 2, 64>;   // 8 waves, 64 x 32
using CfgB = Cfg<128, 96, 4, 2, 1, 2, 64>;    // 8 waves, 32 x 48
using CfgC = Cfg<64, 96, 2, 2, 1, 2, 64>;     // 4 waves, 32 x 48
using CfgE = Cfg<64, 128, 2, 2, 1, 2, 64>;    // 4 waves, 32 x 64
using CfgF = Cfg<64, 64, 2, 2, 1, 3, 64>;     // 4 waves, 32 x 32
// even / odd K order: two wave groups sharing one ring
using SplitC = Cfg<64, 96, 2, 2, 2, 4, 64>;   // 8 waves, 32 x 48
using SplitE = Cfg<64, 128, 2, 2, 2, 4, 64>;
using SplitD = Cfg<128, 128, 2, 2, 2, 4, 64>;
using SplitG = Cfg<32, 64, 1, 2, 2, 4, 64>;   // 4 waves, 32 x 32: small products

enum class Tile { A, D, B, C, E, F, SplitC, SplitE, SplitD, SplitG };

// K summation order from the weight shape (N, K) only: K >= 2048 uses the
// split (even/odd) order, shorter K the sequential order.  So a given weight
// matrix always sums each output in the same order, whatever M (the batch),
// the CU quota or the tile shape -- outputs stay bit-identical across them.
bool split_k_order(int /*N*/, int K) { return K >= 2048; }

long tiles_of(int M, int N, int bm, int bn) { return (long)((M + bm - 1) / bm) * (N / bn); }

// Tile shape.  The K order comes from (N, K) alone (split_k_order) and every
// tile shape of an order adds the same terms in the same sequence, so the
// shape may follow the launch (M, and the n_cu CUs the stream may use)
// without changing a bit.  Sequential order: the largest tile that still
// gives min(256, 2 n_cu) tiles (one per CU of the device, two per CU of a
// share up to 128 CUs); if none does, the one with the most tiles.  Split
// order: 64 x 96 (or 64 x 128 / 128 x 128) tiles, or 32 x 64 ones when the
// product is too small to give three quarters of the CUs a larger tile.  Tile widths
// divide `align` (d_model for the QKV scatter, so that no tile straddles the
// Q / K / V boundaries).
// Work on the share's busiest CU with a bm x bn tile: tiles per CU, rounded
// up, times the tile's area.
long busiest_cu_work(int M, int N, int bm, int bn, int n_cu) {
    return (tiles_of(M, N, bm, bn) + n_cu - 1) / n_cu * (long)bm * bn;
}

// A 128 x 128 tile of the same K order replaces the first choice when it
// leaves the busiest CU with at most 90% of the work: on shares whose CU
// count does not divide the first choice's tiles (192 CUs: 512 tiles of
// 64 x 96 leave some CUs three, 192 tiles of 128 x 128 one each).
bool rebalance_to_128(int M, int N, int align, int n_cu, int bm, int bn) {
    return align % 128 == 0 && 10 * busiest_cu_work(M, N, 128, 128, n_cu) <= 9 * busiest_cu_work(M, N, bm, bn, n_cu);
}

// wide_ok = false skips the 128 x 192 tile: with the LayerNorm-residual
// epilogue it needs more registers than its two workgroups per CU leave and
// spills (at 64 CUs, where it is the first choice for a 768-wide product, the
// 128 x 96 tile is 30% faster).
Tile choose_tile(int M, int N, int K, int align, int n_cu, bool wide_ok = true) {
    if (split_k_order(N, K)) {
        // every split-order product takes a split-order tile: SplitG (64 wide)
        // serves any width the others do not divide, whatever M and n_cu are
        if (align % 96 && align % 128) return Tile::SplitG;
        const bool small = (align % 96 == 0 ? tiles_of(M, N, 64, 96) : tiles_of(M, N, 64, 128)) < 3L * n_cu / 4;
        if (small) return Tile::SplitG;
        if (align % 96 == 0) return rebalance_to_128(M, N, align, n_cu, 64, 96) ? Tile::SplitD : Tile::SplitC;
        if (tiles_of(M, N, 64, 128) < 512) return Tile::SplitE;
        return Tile::SplitD;
    }
    struct Cand { Tile t; int bm, bn; } cands[] = {
        {Tile::A, 128, 192}, {Tile::D, 128, 128}, {Tile::B, 128, 96},
        {Tile::C, 64, 96}, {Tile::E, 64, 128}, {Tile::F, 64, 64}};
    Tile best = Tile::F;
    int best_bm = 64, best_bn = 64;
    long best_n = 0;
    const long enough = std::min(256, 2 * n_cu);   // two tiles per CU on a share of <= 128 CUs
    for (const Cand &c : cands) {
        if (align % c.bn || (!wide_ok && c.t == Tile::A)) continue;
        const long n = tiles_of(M, N, c.bm, c.bn);
        if (n >= enough) {
            best = c.t;
            best_bm = c.bm;
            best_bn = c.bn;
            break;
        }
        if (n > best_n) { best = c.t; best_bm = c.bm; best_bn = c.bn; best_n = n; }
    }
    if (best != Tile::D && rebalance_to_128(M, N, align, n_cu, best_bm, best_bn)) return Tile::D;
    return best;
}

struct TileDims { int bm, bn; bool split; };

template <class C>
constexpr TileDims dims_of() { return {C::BM, C::BN, C::G == 2}; }

TileDims tile_dims(Tile t) {
    switch (t) {
    case Tile::A: return dims_of<CfgA>();
    case Tile::D: return dims_of<CfgD>();
    case Tile::B: return dims_of<CfgB>();
    case Tile::C: return dims_of<CfgC>();
    case Tile::E: return dims_of<CfgE>();
    case Tile::F: return dims_of<CfgF>();
    case Tile::SplitC: return dims_of<SplitC>();
    case Tile::SplitE: return dims_of<SplitE>();
    case Tile::SplitD: return dims_of<SplitD>();
    case Tile::SplitG: return dims_of<SplitG>();
    }
    return {0, 0, false};
}

template <class C>
hipError_t launch_tile(Epi epi, GemmParams &p, hipStream_t s) {
    p.tiles_m = (p.M + C::BM - 1) / C::BM;
    p.tiles_n = p.N / C::BN;
    const dim3 grid(p.tiles_m * p.tiles_n), block(C::NT);
    switch (epi) {
    case Epi::BiasBf16: return launch_kernel(gemm_kernel<C, Epi::BiasBf16>, grid, block, s, p);
    case Epi::BiasGeluBf16: return launch_kernel(gemm_kernel<C, Epi::BiasGeluBf16>, grid, block, s, p);
    case Epi::BiasResidF32: return launch_kernel(gemm_kernel<C, Epi::BiasResidF32>, grid, block, s, p);
    case Epi::Qkv: return launch_kernel(gemm_kernel<C, Epi::Qkv>, grid, block, s, p);
    case Epi::BiasLnResidF32: return launch_kernel(gemm_kernel<C, Epi::BiasLnResidF32>, grid, block, s, p);
    case Epi::F32: return launch_kernel(gemm_kernel<C, Epi::F32>, grid, block, s, p);
    case Epi::GeluBwdBf16: return launch_kernel(gemm_kernel<C, Epi::GeluBwdBf16>, grid, block, s, p);
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------- skinny GEMM (decode)
//
// M <= 16 token rows (one decode step of a batch): the product is bound by
// reading W once, so what matters is how many weight bytes are in flight on
// how many CUs.  A workgroup of 8 waves owns 16 / G output features and the
// whole of K, cut into G equal K-groups that one MFMA works on side by side:
// operand row (g, f) holds feature f's weights of K-group g, operand column
// (g, t) token t's activations of K-group g, and the diagonal blocks of the
// 16 x 16 product (row group == column group) are the per-group partial sums,
// added over g at the end (the off-diagonal blocks are discarded).  G = 1, 2
// or 4 (up to 16 / G tokens) is the largest whose N / (16 / G) workgroups all
// fit the chip at once.  The waves split the K steps (wave w takes w, w + 8,
// ...); each lane loads its weight and activation fragments straight into
// registers (16 bytes each; token columns past M repeat the last row and are
// never stored), as many K steps deep as the wave has, up to 8.  The waves' partial sums are added in wave order through
// LDS, then the K-groups in group order through lane shuffles: the summation
// order depends on K and G only.
//
// With a LayerNorm prologue the activations are LayerNorm(z) of fp32 rows z
// (a pre-LN block's input), normalised by the workgroup itself into LDS as
// bf16 while the first weight fragments are already in flight.  Needs
// M * K <= kSkinnyLnElems and K <= 4096.
//
// Weights come either row-major ([N, K]: one load instruction covers 16 rows
// x 64 bytes) or packed (FRAG): a copy of W in which the 64 lanes' 16-byte
// pieces of one (workgroup, K step) fragment are one contiguous 1 KB block,
// in lane order, blocks ordered by workgroup then K step.  A load instruction
// then reads 1 KB of consecutive addresses, which streams from HBM at the
// rate of a plain copy; the fragments, the MFMAs and the summation order are
// the same in both forms, so the results are bit-identical.  The packed copy
// is specific to one K-group count G (skinny_pack).  The epilogue's operands
// (bias, residual rows) and, without the LayerNorm prologue, the activations
// are requested before the weights, so that no load is left to start after
// the weight stream has ended.
constexpr int kSkinnyWaves = 8, kSkinnyUnroll = 8;
constexpr int kSkinnyLnElems = 16384;
constexpr int kSkinnyCus = 256;              // MI355X compute units

// One wave per row (rows w and w + 8 for wave w), the row held in registers
// (lane l owns the f32x4 vectors l + 64 c).  load() issues the wave's first
// row (waves past the last row load none) and this thread's share of gamma
// and beta -- before the weight fragments, so that they are not queued behind
// them; finish() stages gamma and beta in LDS,
// takes mean and rstd two-pass over the registers with a fixed reduction tree (wave_sum) and
// writes y = fma(gamma, (z - mean) * rstd, beta), rounded to bf16, into the
// activation tile.  NVL = K / 256 rounded up to 8 or 16 (K <= 4096).
// finish() contains one barrier, reached by every wave.
template <int NVL>
struct SkinnyLn {
    static constexpr int GBV = NVL * 64 / (64 * kSkinnyWaves);   // gamma / beta vectors per thread
    f32x4 v[NVL];
    f32x4 g[GBV], b[GBV];

    // Every vector of the row is loaded (indices clamped into the row; the
    // extra vectors are never used), so that the wait for them does not wait
    // for the weights.
    __device__ void load_row(const GemmParams &p, int r, int lane) {
        const f32x4 *zr = reinterpret_cast<const f32x4 *>(p.lnin.z + (size_t)r * p.K);
#pragma unroll
        for (int c = 0; c < NVL; ++c) v[c] = zr[min(c * 64 + lane, p.K / 4 - 1)];
    }

    __device__ void load(const GemmParams &p, int tid, int lane, int wave) {
#pragma unroll
        for (int j = 0; j < GBV; ++j) {
            const int i = min(tid + j * 64 * kSkinnyWaves, p.K / 4 - 1);
            g[j] = reinterpret_cast<const f32x4 *>(p.lnin.gamma)[i];
            b[j] = reinterpret_cast<const f32x4 *>(p.lnin.beta)[i];
        }
        if (wave < p.M) load_row(p, wave, lane);
    }

    __device__ void finish(const GemmParams &p, bf16_t *a_lds, float *gb_lds, int tid, int lane, int wave) {
        const int nv = p.K / 4;
        const float inv_k = 1.0f / (float)p.K;
        f32x4 *g_l = reinterpret_cast<f32x4 *>(gb_lds), *b_l = g_l + nv;
#pragma unroll
        for (int j = 0; j < GBV; ++j) {
            const int i = tid + j * 64 * kSkinnyWaves;
            if (i < nv) {
                g_l[i] = g[j];
                b_l[i] = b[j];
            }
        }
        float mean = 0.f, rstd = 0.f;
        auto stats = [&] {
            float sum = 0.f;
#pragma unroll
            for (int c = 0; c < NVL; ++c)
                if (c * 64 + lane < nv) sum += v[c][0] + v[c][1] + v[c][2] + v[c][3];
            mean = wave_sum(sum) * inv_k;
            float ss = 0.f;
#pragma unroll
            for (int c = 0; c < NVL; ++c)
                if (c * 64 + lane < nv)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float d = v[c][e] - mean;
                        ss += d * d;
                    }
            rstd = 1.0f / sqrtf(wave_sum(ss) * inv_k + p.lnin.eps);
        };
        // gamma and beta of two vectors read before either is used (indices
        // clamped: unused past the row)
        auto emit = [&](int r) {
#pragma unroll
            for (int c = 0; c < NVL; c += 2) {
                f32x4 gg[2], bb[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int i = min((c + h) * 64 + lane, nv - 1);
                    gg[h] = g_l[i];
                    bb[h] = b_l[i];
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int i = (c + h) * 64 + lane;
                    if (i < nv) {
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            y[e] = __builtin_fmaf(gg[h][e], (v[c + h][e] - mean) * rstd, bb[h][e]);
                        *reinterpret_cast<u32x2 *>(a_lds + (size_t)r * p.K + 4 * i) =
                            u32x2{pack2(y[0], y[1]), pack2(y[2], y[3])};
                    }
                }
            }
        };
        if (wave < p.M) stats();
        __syncthreads();                      // gamma and beta staged
        if (wave < p.M) emit(wave);
        if (wave + kSkinnyWaves < p.M) {
            load_row(p, wave + kSkinnyWaves, lane);
            stats();
            emit(wave + kSkinnyWaves);
        }
    }
};

// NVL: 0 = activations from a; 8 or 16 = LayerNorm prologue for K <= 2048 / 4096.
// FRAG: p.w is the packed copy of W (skinny_pack) for this G.  U: K steps a
// wave requests at once (skinny_unroll: the wave's share of the steps, up to 8).
template <Epi EPI, int G, int NVL, bool FRAG, int U>
__global__ __launch_bounds__(64 * kSkinnyWaves) void skinny_kernel(GemmParams p) {
    constexpr bool LNA = NVL > 0;
    constexpr int NW = kSkinnyWaves;
    constexpr int FPW = 16 / G, TPW = 16 / G;      // features and token columns per K-group
    constexpr int kPartBytes = (NW - 1) * 64 * 16;
    // the LayerNorm prologue's bf16 activation tile, later the waves' partial
    // sums; the prologue's gamma and beta (fp32, K each) in an array of their own
    constexpr int kLdsBytes = LNA && kSkinnyLnElems * 2 > kPartBytes ? kSkinnyLnElems * 2 : kPartBytes;
    __shared__ __attribute__((aligned(16))) char lds[kLdsBytes];
    __shared__ __attribute__((aligned(16))) float gb_lds[LNA ? 2 * NVL * 256 : 4];
    f32x4 (*part)[64] = reinterpret_cast<f32x4 (*)[64]>(lds);
    bf16_t *a_lds = reinterpret_cast<bf16_t *>(lds);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.x * FPW;
    const int row = lane & 15, chunk = lane >> 4;               // operand row / column, 8-element K chunk
    const int kg = p.K / G;                                     // K-group length
    const int grp = row / FPW;                                  // K-group of this lane's row and column
    const int wf_row = n0 + row % FPW, a_row = min(row % TPW, p.M - 1);
    const int steps = kg / 32;
    // row-major: step s of this lane at wrow + 32 s; packed: at wrow + 512 s
    constexpr int WSTEP = FRAG ? 512 : 32;
    const bf16_t *wrow = FRAG ? p.w + (size_t)blockIdx.x * steps * 512 + lane * 8
                              : p.w + (size_t)wf_row * p.K + grp * kg + chunk * 8;
    const bf16_t *arow = (LNA ? a_lds : p.a) + (size_t)a_row * p.K + grp * kg + chunk * 8;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    // The epilogue's operands are fetched first.  Lane (fq, t) of wave 0
    // stores features n0 + 4 fq .. + 3 of token t (see below); every lane
    // loads (indices clamped into the operands, no branch), so that no wait
    // for these loads is placed ahead of the weights'.
    const int fq = lane / TPW, t = lane % TPW;
    const bool stores = wave == 0 && lane < (FPW / 4) * TPW && t < p.M;
    const int f_out = n0 + 4 * fq;
    const u32x2 braw = *reinterpret_cast<const u32x2 *>(p.bias + min(f_out, p.N - 4));
    f32x4 rres = {0.f, 0.f, 0.f, 0.f};
    if constexpr (EPI == Epi::BiasResidF32)
        rres = *reinterpret_cast<const f32x4 *>(p.resid + (size_t)min(t, p.M - 1) * p.N + min(f_out, p.N - 4));
    // Fragments past the wave's last K step are replaced by zeros where the
    // MFMA takes them, and every MFMA runs: a skipped step adds exactly zero.
    // (A conditional MFMA may be issued with the wave's EXEC mask empty, which
    // does not stop it from reading its operand registers.)  The selection sits
    // at the MFMA, not at the load, so that no MFMA waits for a later fragment.
    const bf16x8 zero = {};
    bf16x8 wf[U], af[U];
    // Every load is issued, steps past the wave's last one clamped to it
    // (their fragments are zeroed at the MFMA): no branch around a load, so
    // each MFMA waits for its own fragments alone
    auto load_w = [&](int s0) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            wf[u] = *reinterpret_cast<const bf16x8 *>(wrow + min(s0 + u * NW, steps - 1) * WSTEP);
    };
    auto load_a = [&](int s0) {
#pragma unroll
        for (int u = 0; u < U; ++u)
            af[u] = *reinterpret_cast<const bf16x8 *>(arow + min(s0 + u * NW, steps - 1) * 32);
    };
    if constexpr (LNA) {
        // the LayerNorm inputs first, then the weights; the activations are
        // normalised while the weights stream in
        SkinnyLn<NVL> ln;
        ln.load(p, threadIdx.x, lane, wave);
        __builtin_amdgcn_sched_barrier(0);     // keep these loads ahead of the weights' (in-order returns)
        load_w(wave);
        ln.finish(p, a_lds, gb_lds, threadIdx.x, lane, wave);
        __syncthreads();
    } else {
        // the first round's activations (L2-resident) ahead of the weights
        load_a(wave);
        load_w(wave);
    }
    for (int s0 = wave; s0 < steps; s0 += NW * U) {
        if (LNA || s0 != wave) load_a(s0);
#pragma unroll
        for (int u = 0; u < U; ++u)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(s0 + u * NW < steps ? wf[u] : zero,
                                                          s0 + u * NW < steps ? af[u] : zero, acc, 0, 0, 0);
        if (s0 + NW * U < steps) load_w(s0 + NW * U);
    }
    if constexpr (LNA) __syncthreads();                        // the partials reuse the activations' LDS
    if (wave > 0) part[wave - 1][lane] = acc;
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 0; w < NW - 1; ++w) acc += part[w][lane];
    // lane l holds product rows 4 (l / 16) + e, column l % 16.  Output lane
    // (fq, t) gathers features 4 fq .. 4 fq + 3 of token t from the diagonal
    // block of every K-group: row g FPW + 4 fq + e, column g TPW + t.
    if constexpr (G > 1) {
        f32x4 sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int src = (16 * (g * FPW / 4 + fq) + g * TPW + t) & 63;
#pragma unroll
            for (int e = 0; e < 4; ++e) sum[e] += __shfl(acc[e], src);
        }
        acc = sum;
    }
    if (!stores) return;
    const int f = f_out;
    // this lane: features f .. f + 3 of token t
    float v0 = acc[0] + __uint_as_float(braw[0] << 16), v1 = acc[1] + __uint_as_float(braw[0] & 0xffff0000u);
    float v2 = acc[2] + __uint_as_float(braw[1] << 16), v3 = acc[3] + __uint_as_float(braw[1] & 0xffff0000u);
    if constexpr (EPI == Epi::BiasBf16 || EPI == Epi::BiasGeluBf16) {
        if constexpr (EPI == Epi::BiasGeluBf16) {
            v0 = gelu(v0); v1 = gelu(v1); v2 = gelu(v2); v3 = gelu(v3);
        }
        *reinterpret_cast<u32x2 *>(static_cast<bf16_t *>(p.out) + (size_t)t * p.N + f) =
            u32x2{pack2(v0, v1), pack2(v2, v3)};
    } else if constexpr (EPI == Epi::BiasResidF32) {
        const f32x4 r = rres;
        *reinterpret_cast<f32x4 *>(static_cast<float *>(p.out) + (size_t)t * p.N + f) =
            f32x4{r[0] + v0, r[1] + v1, r[2] + v2, r[3] + v3};
    } else if constexpr (EPI == Epi::Qkv) {
        const QkvDst &d = p.qkv;
        const int which = f / d.d_model, within = f - which * d.d_model;
        const int head = within / d.head_dim, jj = within - head * d.head_dim;
        const int b = t / d.seq, sp = t - b * d.seq;
        const size_t bh = (size_t)b * d.n_heads + head;
        if (which < 2) {
            bf16_t *o = which == 0 ? d.q + (bh * d.seq + sp) * d.head_dim + jj
                                   : d.k + (bh * d.k_rows + d.pos0 + sp) * d.head_dim + jj;
            *reinterpret_cast<u32x2 *>(o) = u32x2{pack2(v0, v1), pack2(v2, v3)};
        } else {
            bf16_t *o = d.vt + (bh * d.head_dim + jj) * d.vt_stride + d.pos0 + sp;
            o[0] = f32_to_bf16(v0);
            o[d.vt_stride] = f32_to_bf16(v1);
            o[2 * (size_t)d.vt_stride] = f32_to_bf16(v2);
            o[3 * (size_t)d.vt_stride] = f32_to_bf16(v3);
        }
    }
}

}  // namespace

GemmPlan gemm_plan(int M, int N, int K, int align, int n_cu, bool ln_residual) {
    const TileDims d = tile_dims(choose_tile(M, N, K, align, n_cu, !ln_residual));
    return GemmPlan{split_k_order(N, K), d.split, d.bm, d.bn};
}

hipError_t launch_gemm(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                       const float *resid, void *out, int M, int N, int K, const QkvDst *qkv,
                       hipStream_t stream, const LnResid *ln, const bf16_t *aux, int n_cu) {
    if (M <= 0) return hipSuccess;
    if (N % 64 || K % 64 || N <= 0 || K <= 0) return hipErrorInvalidValue;
    if (epi == Epi::GeluBwdBf16 && !aux) return hipErrorInvalidValue;
    GemmParams p{};
    p.a = a; p.w = w; p.bias = bias; p.resid = resid; p.out = out; p.aux = aux;
    p.M = M; p.N = N; p.K = K;
    if (qkv) p.qkv = *qkv;
    if (ln) p.ln = *ln;
    // N is a multiple of 64 (checked by the callers); d_model a multiple of 128
    const int align = epi == Epi::Qkv ? p.qkv.d_model : N;
    switch (choose_tile(M, N, K, align, n_cu, epi != Epi::BiasLnResidF32)) {
    case Tile::A: return launch_tile<CfgA>(epi, p, stream);
    case Tile::D: return launch_tile<CfgD>(epi, p, stream);
    case Tile::B: return launch_tile<CfgB>(epi, p, stream);
    case Tile::C: return launch_tile<CfgC>(epi, p, stream);
    case Tile::E: return launch_tile<CfgE>(epi, p, stream);
    case Tile::F: return launch_tile<CfgF>(epi, p, stream);
    case Tile::SplitC: return launch_tile<SplitC>(epi, p, stream);
    case Tile::SplitE: return launch_tile<SplitE>(epi, p, stream);
    case Tile::SplitD: return launch_tile<SplitD>(epi, p, stream);
    case Tile::SplitG: return launch_tile<SplitG>(epi, p, stream);
    }
    return hipErrorInvalidValue;
}

namespace {

template <int G, int NVL, bool FRAG, int U>
hipError_t launch_skinny(Epi epi, const GemmParams &p, hipStream_t stream) {
    const dim3 grid(p.N / (16 / G)), block(64 * kSkinnyWaves);
    switch (epi) {
    case Epi::BiasBf16: return launch_kernel(skinny_kernel<Epi::BiasBf16, G, NVL, FRAG, U>, grid, block, stream, p);
    case Epi::BiasGeluBf16:
        return launch_kernel(skinny_kernel<Epi::BiasGeluBf16, G, NVL, FRAG, U>, grid, block, stream, p);
    case Epi::BiasResidF32:
        return launch_kernel(skinny_kernel<Epi::BiasResidF32, G, NVL, FRAG, U>, grid, block, stream, p);
    case Epi::Qkv: return launch_kernel(skinny_kernel<Epi::Qkv, G, NVL, FRAG, U>, grid, block, stream, p);
    case Epi::BiasLnResidF32:
    case Epi::F32:
    case Epi::GeluBwdBf16: break;
    }
    return hipErrorInvalidValue;
}

// K steps a wave requests at once: its share of the product's steps, rounded
// up to a power of two, at most kSkinnyUnroll (more steps take more rounds)
int skinny_unroll(int K, int G) {
    const int per_wave = (K / G / 32 + kSkinnyWaves - 1) / kSkinnyWaves;
    int u = 1;
    while (u < per_wave && u < kSkinnyUnroll) u *= 2;
    return u;
}

template <int G, int NVL, bool FRAG>
hipError_t launch_skinny_u(Epi epi, const GemmParams &p, hipStream_t stream) {
    switch (skinny_unroll(p.K, G)) {
    case 1: return launch_skinny<G, NVL, FRAG, 1>(epi, p, stream);
    case 2: return launch_skinny<G, NVL, FRAG, 2>(epi, p, stream);
    case 4: return launch_skinny<G, NVL, FRAG, 4>(epi, p, stream);
    default: return launch_skinny<G, NVL, FRAG, 8>(epi, p, stream);
    }
}

template <int NVL>
hipError_t launch_skinny_g(Epi epi, const GemmParams &p, int g, bool frag, hipStream_t stream) {
    switch (g) {
    case 1: return frag ? launch_skinny_u<1, NVL, true>(epi, p, stream) : launch_skinny_u<1, NVL, false>(epi, p, stream);
    case 2: return frag ? launch_skinny_u<2, NVL, true>(epi, p, stream) : launch_skinny_u<2, NVL, false>(epi, p, stream);
    case 4: return frag ? launch_skinny_u<4, NVL, true>(epi, p, stream) : launch_skinny_u<4, NVL, false>(epi, p, stream);
    }
    return hipErrorInvalidValue;
}

// Packed copy for the skinny product with G K-groups: 16-byte piece i of dst
// is what lane l of workgroup b loads at K step s in the row-major form, with
// i = (b * steps + s) * 64 + l; steps = K / (32 G).
template <int G>
__global__ __launch_bounds__(256) void skinny_pack_kernel(const bf16_t *w, bf16_t *dst, int N, int K) {
    constexpr int FPW = 16 / G;
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const int kg = K / G, steps = kg / 32;
    if (i >= (size_t)N * K / 8) return;
    const int l = (int)(i % 64);
    const size_t bs = i / 64;
    const int s = (int)(bs % steps), b = (int)(bs / steps);
    const int row = l & 15, chunk = l >> 4;
    const int f = b * FPW + row % FPW, grp = row / FPW;
    const size_t k = (size_t)grp * kg + s * 32 + chunk * 8;
    reinterpret_cast<bf16x8 *>(dst)[i] = *reinterpret_cast<const bf16x8 *>(w + (size_t)f * K + k);
}

}  // namespace

int skinny_groups(int M, int N, int K, bool ln) {
    // more K-groups while the workgroups still fit the CUs in one round (3 per
    // CU, 2 with the LayerNorm prologue's registers and LDS), so that no
    // workgroup starts streaming its weights only after another has finished
    const int limit = (ln ? 2 : 3) * kSkinnyCus;
    int g = 1;
    while (g < 4 && N / (16 / (2 * g)) <= limit && M <= 16 / (2 * g) && K % (32 * 2 * g) == 0) g *= 2;
    return g;
}

bool skinny_ln_fits(int M, int K) {
    return M >= 1 && M <= 16 && K % 32 == 0 && K <= 4096 && M * K <= kSkinnyLnElems;
}

hipError_t launch_skinny_pack(const bf16_t *w, bf16_t *dst, int N, int K, int groups, hipStream_t stream) {
    if (N <= 0 || K <= 0 || (groups != 1 && groups != 2 && groups != 4)) return hipErrorInvalidValue;
    if (N % (16 / groups) || K % (32 * groups)) return hipErrorInvalidValue;
    const size_t pieces = (size_t)N * K / 8;
    const dim3 grid((unsigned)((pieces + 255) / 256)), block(256);
    switch (groups) {
    case 1: return launch_kernel(skinny_pack_kernel<1>, grid, block, stream, w, dst, N, K);
    case 2: return launch_kernel(skinny_pack_kernel<2>, grid, block, stream, w, dst, N, K);
    default: return launch_kernel(skinny_pack_kernel<4>, grid, block, stream, w, dst, N, K);
    }
}

hipError_t launch_gemm_skinny(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias, const float *resid,
                              void *out, int M, int N, int K, const QkvDst *qkv, hipStream_t stream,
                              const LnIn *ln_in, const bf16_t *w_packed, int packed_groups) {
    if (M <= 0) return hipSuccess;
    if (M > 16 || N % 16 || K % 32 || epi == Epi::BiasLnResidF32 || epi == Epi::F32 || epi == Epi::GeluBwdBf16)
        return hipErrorInvalidValue;
    if (ln_in && !skinny_ln_fits(M, K)) return hipErrorInvalidValue;
    GemmParams p{};
    p.a = a; p.w = w; p.bias = bias; p.resid = resid; p.out = out;
    p.M = M; p.N = N; p.K = K;
    if (qkv) p.qkv = *qkv;
    if (ln_in) p.lnin = *ln_in;
    const int g = skinny_groups(M, N, K, ln_in != nullptr);
    const bool frag = w_packed && packed_groups == g;
    if (frag) p.w = w_packed;
    if (!ln_in) return launch_skinny_g<0>(epi, p, g, frag, stream);
    return K <= 2048 ? launch_skinny_g<8>(epi, p, g, frag, stream) : launch_skinny_g<16>(epi, p, g, frag, stream);
}

}  // namespace iefwd
