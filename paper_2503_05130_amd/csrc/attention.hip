// Fused softmax attention for gfx950: ctx = softmax(Q K^T / sqrt(dh) [+ causal]) V
// per (batch, head), with an online softmax over 32-key blocks.
//
// Work split.  A workgroup of 4 waves owns 128 queries of one (batch, head);
// each wave owns 32 of them.  Keys are streamed in 64-key chunks: the whole
// workgroup copies a chunk of K ([64, dh]) and of V^T ([dh, 64]) from global
// memory into LDS (double-buffered, the next chunk's global loads in flight
// while the current chunk is consumed), so each K/V element is fetched from
// L2/HBM once per workgroup instead of once per wave.
//
// Layout trick.  Each wave computes the *transposed* score block S^T = K Q^T
// (keys x queries) with v_mfma_f32_32x32x16_bf16.  In the 32x32 accumulator
// layout lane l holds column l % 32 -- one query -- and 16 of the 32 keys (the
// other 16 sit in lane l ^ 32).  So:
//   * the softmax row max / row sum are in-register reductions plus one
//     exchange with lane l ^ 32;
//   * the online-softmax rescale factor is per lane: rescaling the context
//     accumulator needs no cross-lane traffic;
//   * the probabilities, converted to bf16 in place, are directly the "B"
//     operand of ctx^T = V^T P^T: an MFMA contracts over whatever k order its
//     two operands agree on, so V^T is read in the key order the accumulator
//     layout already has (keys 4h..4h+3 and 8+4h..8+4h+3 of each 16-key step,
//     h = lane / 32).
// V is stored transposed, [B, H, dh, S_pad] (S_pad = S rounded up to 64), by
// the QKV epilogue, so every fragment is a contiguous 16- or 8-byte read.
//
// Precision: scores, softmax and the accumulator are fp32; P is rounded to bf16
// for the PV product; ctx is rounded to bf16 (the out-projection's operand).
// Determinism: fixed key-block order, fixed reduction tree, no atomics.
#include "kernels.h"

namespace iefwd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;          // 4 waves x 32 queries = 128 queries per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kChunk = 64;         // keys per LDS chunk
constexpr int kVtStride = kChunk + 8;   // V^T chunk row (bf16): 144 bytes

__device__ inline uint16_t to_bf16_bits(float f) {
    __bf16 b = (__bf16)f;
    return __builtin_bit_cast(uint16_t, b);
}

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int DH, bool CAUSAL>
__global__ __launch_bounds__(kThreads) void attention_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ Vt,
    bf16_t *__restrict__ ctx, int n_heads, int seq, int k_rows, int seq_pad, float scale_log2e) {
    constexpr int KS = DH / 16;              // 16-wide k steps of the QK^T product
    constexpr int DB = DH / 32;              // 32-row dh blocks of the context accumulator
    constexpr int K_STRIDE = DH + 8;         // K chunk row (bf16): 16 consecutive rows in distinct banks
    constexpr int K_ELEMS = kChunk * K_STRIDE;
    constexpr int V_ELEMS = DH * kVtStride;
    constexpr int K_CH = kChunk * (DH / 8) / kThreads;   // 16-byte pieces per thread per chunk
    constexpr int V_CH = DH * (kChunk / 8) / kThreads;
    static_assert(K_CH >= 1 && V_CH >= 1, "chunk split");

    __shared__ __attribute__((aligned(16))) bf16_t lds[2 * (K_ELEMS + V_ELEMS)];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, col = lane & 31;
    // heaviest query groups first when causal (they see the most keys)
    const int qgroup = CAUSAL ? (int)(gridDim.x - 1 - blockIdx.x) : (int)blockIdx.x;
    const int qg0 = qgroup * 32 * kWaves;
    const int q0 = qg0 + wave * 32;                      // this wave's first query
    const int bh = blockIdx.y;
    const bf16_t *Qh = Q + (size_t)bh * seq * DH;
    const bf16_t *Kh = K + (size_t)bh * k_rows * DH;
    const bf16_t *Vh = Vt + (size_t)bh * DH * seq_pad;

    const int query = q0 + col;
    const bool wave_active = q0 < seq;                   // waves past the end still help load
    const int q_row = min(query, seq - 1);

    bf16x8 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
        qf[ks] = as_bf16x8(*reinterpret_cast<const u32x4 *>(Qh + (size_t)q_row * DH + ks * 16 + half * 8));

    f32x16 acc[DB];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[d][r] = 0.f;
    float m_run = -INFINITY;   // running max (log2 domain), shared by both halves
    float l_run = 0.f;         // this half's running sum of probabilities

    // keys this workgroup needs: all of them, or up to its last query when causal
    const int key_end = CAUSAL ? min(qg0 + 32 * kWaves, seq) : seq;
    const int n_chunks = (key_end + kChunk - 1) / kChunk;
    const int wave_key_end = CAUSAL ? min(q0 + 32, seq) : seq;   // this wave's visible keys

    // cooperative chunk copy: global -> registers -> LDS
    u32x4 kreg[K_CH], vreg[V_CH];
    auto gload = [&](int c) {
        const int k0 = c * kChunk;
#pragma unroll
        for (int i = 0; i < K_CH; ++i) {
            const int piece = tid + i * kThreads;
            const int row = piece / (DH / 8), cp = piece % (DH / 8);
            const int key = min(k0 + row, seq - 1);             // clamped: finite, masked later
            kreg[i] = *reinterpret_cast<const u32x4 *>(Kh + (size_t)key * DH + cp * 8);
        }
#pragma unroll
        for (int i = 0; i < V_CH; ++i) {
            const int piece = tid + i * kThreads;
            const int row = piece / (kChunk / 8), cp = piece % (kChunk / 8);
            u32x4 v = *reinterpret_cast<const u32x4 *>(Vh + (size_t)row * seq_pad + k0 + cp * 8);
            const int kfirst = k0 + cp * 8;
            if (kfirst + 8 > seq) {   // padding past seq holds arbitrary bits: zero it (P is 0 there)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] &= (kfirst + 2 * e < seq ? 0x0000ffffu : 0u) | (kfirst + 2 * e + 1 < seq ? 0xffff0000u : 0u);
            }
            vreg[i] = v;
        }
    };
    auto lstore = [&](int buf) {
        bf16_t *kb = lds + buf * (K_ELEMS + V_ELEMS);
        bf16_t *vb = kb + K_ELEMS;
#pragma unroll
        for (int i = 0; i < K_CH; ++i) {
            const int piece = tid + i * kThreads;
            const int row = piece / (DH / 8), cp = piece % (DH / 8);
            *reinterpret_cast<u32x4 *>(kb + row * K_STRIDE + cp * 8) = kreg[i];
        }
#pragma unroll
        for (int i = 0; i < V_CH; ++i) {
            const int piece = tid + i * kThreads;
            const int row = piece / (kChunk / 8), cp = piece % (kChunk / 8);
            *reinterpret_cast<u32x4 *>(vb + row * kVtStride + cp * 8) = vreg[i];
        }
    };

    gload(0);
    lstore(0);
    __syncthreads();
    for (int c = 0; c < n_chunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < n_chunks) gload(c + 1);
        const bf16_t *kb = lds + buf * (K_ELEMS + V_ELEMS);
        const bf16_t *vb = kb + K_ELEMS;
#pragma unroll
        for (int sb = 0; sb < kChunk / 32; ++sb) {
            const int k0 = c * kChunk + sb * 32;
            if (!wave_active || k0 >= wave_key_end) continue;   // wave-uniform
            // ---- S^T block (32 keys x 32 queries)
            f32x16 st;
#pragma unroll
            for (int r = 0; r < 16; ++r) st[r] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4 *>(
                    kb + (sb * 32 + col) * K_STRIDE + ks * 16 + half * 8));
                st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], st, 0, 0, 0);
            }
            // key of accumulator entry r: k0 + 8 (r / 4) + 4 half + r % 4.  Only the
            // diagonal block (causal) or the ragged last block needs the mask.
            const bool need_mask = CAUSAL ? (k0 + 31 > q0) : (k0 + 32 > seq);   // wave-uniform
            float mx = -INFINITY;
            if (need_mask) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = k0 + 8 * (r >> 2) + 4 * half + (r & 3);
                    const bool ok = key < seq && (!CAUSAL || key <= query);
                    st[r] = ok ? st[r] * scale_log2e : -INFINITY;
                    mx = fmaxf(mx, st[r]);
                }
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    st[r] *= scale_log2e;
                    mx = fmaxf(mx, st[r]);
                }
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx);   // finite: key 0 is visible to every query
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            float psum = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                st[r] = __builtin_amdgcn_exp2f(st[r] - m_new);
                psum += st[r];
            }
            l_run = l_run * alpha + psum;
            m_run = m_new;
#pragma unroll
            for (int d = 0; d < DB; ++d)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[d][r] *= alpha;
            // ---- ctx^T += V^T P^T, two 16-key steps
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                bf16x8 pf;   // P^T fragment: entries r = 8 j .. 8 j + 7
#pragma unroll
                for (int e = 0; e < 8; ++e) pf[e] = (__bf16)st[8 * j + e];
                const int kl = sb * 32 + 16 * j + 4 * half;   // chunk-local keys kl..kl+3, kl+8..kl+11
#pragma unroll
                for (int d = 0; d < DB; ++d) {
                    const bf16_t *vrow = vb + (d * 32 + col) * kVtStride;
                    const u32x2 lo = *reinterpret_cast<const u32x2 *>(vrow + kl);
                    const u32x2 hi = *reinterpret_cast<const u32x2 *>(vrow + kl + 8);
                    const u32x4 v = {lo[0], lo[1], hi[0], hi[1]};
                    acc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(v), pf, acc[d], 0, 0, 0);
                }
            }
        }
        if (c + 1 < n_chunks) lstore(buf ^ 1);
        __syncthreads();
    }

    if (!wave_active || query >= seq) return;
    const float inv = 1.f / (l_run + __shfl_xor(l_run, 32));
    // acc[d] entry r is dh index 32 d + 8 (r / 4) + 4 half + r % 4 of this query
    const int h = bh % n_heads, b = bh / n_heads;
    bf16_t *out = ctx + ((size_t)b * seq + query) * (size_t)(n_heads * DH) + h * DH;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int e = 32 * d + 8 * g + 4 * half;
            const uint32_t w0 = (uint32_t)to_bf16_bits(acc[d][4 * g] * inv) |
                                ((uint32_t)to_bf16_bits(acc[d][4 * g + 1] * inv) << 16);
            const uint32_t w1 = (uint32_t)to_bf16_bits(acc[d][4 * g + 2] * inv) |
                                ((uint32_t)to_bf16_bits(acc[d][4 * g + 3] * inv) << 16);
            *reinterpret_cast<u32x2 *>(out + e) = u32x2{w0, w1};
        }
}

template <int DH, bool CAUSAL>
hipError_t launch(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx, int batch,
                  int n_heads, int seq, int k_rows, int vt_stride, hipStream_t s) {
    const int groups = (seq + 32 * kWaves - 1) / (32 * kWaves);
    const dim3 grid(groups, batch * n_heads), block(kThreads);
    const float scale_log2e = 1.4426950408889634f / sqrtf((float)DH);
    return launch_kernel(attention_kernel<DH, CAUSAL>, grid, block, s, q, k, vt, ctx, n_heads, seq, k_rows,
                         vt_stride, scale_log2e);
}

}  // namespace

hipError_t launch_attention(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx,
                            int batch, int n_heads, int seq, int head_dim, bool causal,
                            hipStream_t stream, int k_rows, int vt_stride) {
    if (batch <= 0 || seq <= 0) return hipSuccess;
    if (k_rows <= 0) k_rows = seq;
    if (vt_stride <= 0) vt_stride = attn_seq_pad(seq);
    if (k_rows < seq || vt_stride < attn_seq_pad(seq) || vt_stride % 64 != 0) return hipErrorInvalidValue;
    if (head_dim == 64)
        return causal ? launch<64, true>(q, k, vt, ctx, batch, n_heads, seq, k_rows, vt_stride, stream)
                      : launch<64, false>(q, k, vt, ctx, batch, n_heads, seq, k_rows, vt_stride, stream);
    if (head_dim == 128)
        return causal ? launch<128, true>(q, k, vt, ctx, batch, n_heads, seq, k_rows, vt_stride, stream)
                      : launch<128, false>(q, k, vt, ctx, batch, n_heads, seq, k_rows, vt_stride, stream);
    return hipErrorInvalidValue;
}

}  // namespace iefwd
