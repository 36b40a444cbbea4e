// Decode-phase attention for gfx950: one new query per (batch, head) against
// the keys 0 .. n_keys - 1 of a KV cache.  Memory-bound: every cached K and V
// element is read once, nothing else of size.
//
// One workgroup (4 waves) per (batch, head):
//   1. scores: a key row of K (dh bf16, 16-byte pieces) is read by dh / 8
//      consecutive lanes, each multiplying its 8 elements with the matching
//      part of q; a butterfly over those lanes sums the row.  Scores (times
//      log2 e / sqrt(dh)) go to LDS.
//   2. max and sum over the scores (wave butterflies, then across waves in LDS);
//      the probabilities p_j = 2^(s_j - max) replace the scores in LDS.
//   3. context: V is cached transposed, [dh, positions], so row d of V^T is
//      contiguous over the keys: a wave reads 512 keys of one row per load
//      (8 per lane), multiplies with p_j and reduces; ctx[d] = sum / l.
// Positions past n_keys of the cache may hold any bits: they are never
// multiplied (masked, not zeroed by arithmetic).
//
// Precision: fp32 scores, softmax and sums; q, K, V are bf16 as stored; the
// context is rounded to bf16 (the out-projection's operand).  Determinism:
// fixed assignment of keys to lanes and fixed reduction trees.
#include "kernels.h"

namespace iefwd {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxKeys = 8192;

__device__ inline float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ inline float dot8(u32x4 a, const float (&q)[8]) {
    float s = lo_bf16(a[0]) * q[0];
    s = fmaf(hi_bf16(a[0]), q[1], s);
    s = fmaf(lo_bf16(a[1]), q[2], s);
    s = fmaf(hi_bf16(a[1]), q[3], s);
    s = fmaf(lo_bf16(a[2]), q[4], s);
    s = fmaf(hi_bf16(a[2]), q[5], s);
    s = fmaf(lo_bf16(a[3]), q[6], s);
    s = fmaf(hi_bf16(a[3]), q[7], s);
    return s;
}

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ inline uint16_t to_bf16_bits(float f) {
    __bf16 b = (__bf16)f;
    return __builtin_bit_cast(uint16_t, b);
}

template <int DH>
__global__ __launch_bounds__(kThreads) void decode_attention_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ Vt,
    bf16_t *__restrict__ ctx, int n_heads, int n_keys, int k_rows, int vt_stride, float scale_log2e) {
    constexpr int LPK = DH / 8;               // lanes per key row
    constexpr int KPW = 64 / LPK;             // keys per wave per load
    __shared__ float sc[kMaxKeys];
    __shared__ float red[2 * kWaves];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.x;
    const bf16_t *Kh = K + (size_t)bh * k_rows * DH;
    const bf16_t *Vh = Vt + (size_t)bh * DH * vt_stride;

    // this lane's 8 elements of q
    const int part = lane % LPK;
    float q[8];
    {
        const u32x4 w = *reinterpret_cast<const u32x4 *>(Q + (size_t)bh * DH + part * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            q[2 * e] = lo_bf16(w[e]);
            q[2 * e + 1] = hi_bf16(w[e]);
        }
    }

    // 1. scores
    float mx = -INFINITY;
    for (int base = wave * KPW; base < n_keys; base += kWaves * KPW) {
        const int j = base + lane / LPK;
        const int jr = min(j, n_keys - 1);                  // clamped: in range, result unused
        float s = dot8(*reinterpret_cast<const u32x4 *>(Kh + (size_t)jr * DH + part * 8), q);
#pragma unroll
        for (int o = LPK / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o);
        s *= scale_log2e;
        if (part == 0 && j < n_keys) sc[j] = s;
        if (j < n_keys) mx = fmaxf(mx, s);
    }
    mx = wave_max(mx);
    if (lane == 0) red[wave] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mx = fmaxf(mx, red[w]);

    // 2. probabilities and their sum
    float sum = 0.f;
    for (int j = tid; j < n_keys; j += kThreads) {
        const float p = __builtin_amdgcn_exp2f(sc[j] - mx);
        sc[j] = p;
        sum += p;
    }
    sum = wave_sum(sum);
    __syncthreads();                                       // every wave has read red[] and written sc[]
    if (lane == 0) red[kWaves + wave] = sum;
    __syncthreads();
    float l = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) l += red[kWaves + w];
    const float inv = 1.0f / l;

    // 3. context: rows d = wave, wave + 4, ... of V^T
    for (int d = wave; d < DH; d += kWaves) {
        const bf16_t *row = Vh + (size_t)d * vt_stride;
        float acc = 0.f;
        for (int j0 = lane * 8; j0 < n_keys; j0 += 512) {
            const u32x4 w = *reinterpret_cast<const u32x4 *>(row + j0);
            if (j0 + 8 <= n_keys) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc = fmaf(sc[j0 + 2 * e], lo_bf16(w[e]), acc);
                    acc = fmaf(sc[j0 + 2 * e + 1], hi_bf16(w[e]), acc);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (j0 + 2 * e < n_keys) acc = fmaf(sc[j0 + 2 * e], lo_bf16(w[e]), acc);
                    if (j0 + 2 * e + 1 < n_keys) acc = fmaf(sc[j0 + 2 * e + 1], hi_bf16(w[e]), acc);
                }
            }
        }
        acc = wave_sum(acc);
        if (lane == 0) {
            const int b = bh / n_heads, h = bh - b * n_heads;
            ctx[(size_t)b * n_heads * DH + (size_t)h * DH + d] = to_bf16_bits(acc * inv);
        }
    }
}

}  // namespace

hipError_t launch_decode_attention(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx, int batch,
                                   int n_heads, int n_keys, int head_dim, int k_rows, int vt_stride,
                                   hipStream_t stream) {
    if (batch <= 0) return hipSuccess;
    if (n_keys <= 0 || n_keys > kMaxKeys || k_rows < n_keys || vt_stride < n_keys || vt_stride % 64 != 0)
        return hipErrorInvalidValue;
    const dim3 grid(batch * n_heads), block(kThreads);
    if (head_dim == 64)
        return launch_kernel(decode_attention_kernel<64>, grid, block, stream, q, k, vt, ctx, n_heads, n_keys,
                             k_rows, vt_stride, 1.4426950408889634f / 8.0f);
    if (head_dim == 128)
        return launch_kernel(decode_attention_kernel<128>, grid, block, stream, q, k, vt, ctx, n_heads, n_keys,
                             k_rows, vt_stride, 1.4426950408889634f / sqrtf(128.0f));
    return hipErrorInvalidValue;
}

}  // namespace iefwd
