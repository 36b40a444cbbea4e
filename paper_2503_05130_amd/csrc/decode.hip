// Decode-phase attention for gfx950: one new query per (batch, head) against
// the keys 0 .. n_keys - 1 of a KV cache.  Memory-bound: every cached K and V
// element is read once, nothing else of size.
//
// The keys are split into chunks of CH (64 up to 2048 keys, else 256; at most
// 32 chunks); a workgroup (4 waves) takes one chunk of one (batch, head), so a
// decode step of a few sequences still has enough workgroups to keep HBM busy:
//   1. scores: a key row of K (dh bf16) is read by dh / 8 consecutive lanes,
//      16 bytes each, all of the chunk's rows issued before any is used; a
//      butterfly over those lanes sums the row.  Scores (times log2 e /
//      sqrt(dh)) go to LDS.
//   2. the chunk's max m_c, p_j = 2^(s_j - m_c) and their sum l_c.
//   3. the chunk's context: V is cached transposed, [dh, positions], so a V^T
//      row is contiguous over the chunk's keys: CH / 8 lanes read one row (8
//      keys each), multiply with p_j and reduce.  (m_c, l_c, acc_c[dh]) go to
//      the chunk's slot of a partials buffer.
//   4. a second kernel combines the chunks of each (batch, head):
//      M = max m_c, ctx = sum_c 2^(m_c - M) acc_c / sum_c 2^(m_c - M) l_c, in
//      chunk order.  (Handing the partials over at the kernel boundary keeps
//      the workgroups free of device-scope fences, which on this chip write
//      back and invalidate a whole XCD L2 each.)  A single chunk writes its
//      context directly and needs no second kernel.  The chunking depends on
//      n_keys alone, so a sequence's result depends neither on the batch nor
//      on the CUs used.
// Positions past n_keys of the cache may hold any bits: they are never
// multiplied (masked, not zeroed by arithmetic).
//
// Precision: fp32 scores, softmax and sums; q, K, V are bf16 as stored; the
// context is rounded to bf16 (the out-projection's operand).
#include "kernels.h"

namespace iefwd {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxKeys = 8192;
constexpr int kSmallChunk = 64, kLargeChunk = 256, kSmallLimit = 2048;

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

template <int DH, int CH>
__global__ __launch_bounds__(kThreads) void decode_attention_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ Vt,
    bf16_t *__restrict__ ctx, float *__restrict__ partials, int n_keys, int k_rows, int vt_stride,
    float scale_log2e) {
    constexpr int LPK = DH / 8;                  // lanes per key row of K
    constexpr int KPI = kThreads / LPK;          // key rows per workgroup load
    constexpr int NLOAD = CH / KPI;              // K loads per thread
    constexpr int LPR = CH / 8;                  // lanes per V^T row
    constexpr int RPP = kThreads / LPR;          // V^T rows per pass
    constexpr int SLOT = DH + 2;                 // floats per chunk slot: m, l, acc[DH]
    static_assert(NLOAD >= 1 && CH <= kThreads && DH % RPP == 0, "chunk shape");
    __shared__ float sc[CH];
    __shared__ float red[2 * kWaves];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int chunk = blockIdx.x, n_chunks = gridDim.x, bh = blockIdx.y;
    const int j0 = chunk * CH, nk = min(CH, n_keys - j0);     // this chunk's keys
    const bf16_t *Kh = K + (size_t)bh * k_rows * DH;
    const bf16_t *Vh = Vt + (size_t)bh * DH * vt_stride;

    // this lane's 8 elements of q
    const int part = tid % LPK;
    float q[8];
    {
        const u32x4 w = *reinterpret_cast<const u32x4 *>(Q + (size_t)bh * DH + part * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            q[2 * e] = lo_bf16(w[e]);
            q[2 * e + 1] = hi_bf16(w[e]);
        }
    }

    // 1. scores: all loads first (rows past n_keys are clamped to the last key:
    // read, never used), and with them the V^T rows of step 3, which depend on
    // nothing computed here: one memory round trip for the whole chunk
    u32x4 kr[NLOAD];
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
        const int j = min(j0 + i * KPI + tid / LPK, n_keys - 1);
        kr[i] = *reinterpret_cast<const u32x4 *>(Kh + (size_t)j * DH + part * 8);
    }
    const int r_in = tid / LPR, kk = (tid % LPR) * 8;
    const int kread = min(j0 + kk, vt_stride - 8);    // 16-byte aligned, inside the row; masked below
    u32x4 vr[DH / RPP];
#pragma unroll
    for (int i = 0; i < DH / RPP; ++i)
        vr[i] = *reinterpret_cast<const u32x4 *>(Vh + (size_t)(i * RPP + r_in) * vt_stride + kread);
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
        const int jl = i * KPI + tid / LPK;      // key within the chunk
        float s = dot8(kr[i], q);
#pragma unroll
        for (int o = LPK / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o);
        s *= scale_log2e;
        if (jl < nk) {
            if (part == 0) sc[jl] = s;
            mx = fmaxf(mx, s);
        }
    }
    mx = wave_max(mx);
    if (lane == 0) red[wave] = mx;
    __syncthreads();
    mx = red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) mx = fmaxf(mx, red[w]);

    // 2. probabilities and their sum
    float p = 0.f;
    if (tid < nk) {
        p = __builtin_amdgcn_exp2f(sc[tid] - mx);
        sc[tid] = p;
    }
    const float wsum = wave_sum(p);
    if (lane == 0) red[kWaves + wave] = wsum;
    __syncthreads();
    float l = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) l += red[kWaves + w];

    // 3. the chunk's context: RPP rows of V^T per pass, LPR lanes x 8 keys per row
    float pk[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pk[e] = kk + e < nk ? sc[kk + e] : 0.f;
    const bool single = n_chunks == 1;
    float *slot = partials + ((size_t)bh * n_chunks + chunk) * SLOT;
    const float inv_l = 1.0f / l;
#pragma unroll
    for (int i = 0; i < DH / RPP; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (kk + 2 * e < nk) acc = fmaf(pk[2 * e], lo_bf16(vr[i][e]), acc);
            if (kk + 2 * e + 1 < nk) acc = fmaf(pk[2 * e + 1], hi_bf16(vr[i][e]), acc);
        }
#pragma unroll
        for (int o = LPR / 2; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
        if (tid % LPR == 0) {
            const int dd = i * RPP + r_in;
            if (single)
                ctx[(size_t)bh * DH + dd] = to_bf16_bits(acc * inv_l);
            else
                slot[2 + dd] = acc;
        }
    }
    if (tid == 0 && !single) {
        slot[0] = mx;
        slot[1] = l;
    }
}

// 4. one workgroup of DH threads per (batch, head): the chunks' weights from
// their maxima, then every context element summed over the chunks in order.
// Every partial this thread needs is requested before the first is used.
template <int DH>
__global__ __launch_bounds__(DH) void decode_combine_kernel(const float *__restrict__ partials,
                                                            bf16_t *__restrict__ ctx, int n_chunks) {
    constexpr int SLOT = DH + 2;
    __shared__ float wc[kDecodeMaxChunks];
    __shared__ float lsum;
    const int tid = threadIdx.x, bh = blockIdx.x;
    const float *slots = partials + (size_t)bh * n_chunks * SLOT;
    float part[kDecodeMaxChunks];
#pragma unroll
    for (int c = 0; c < kDecodeMaxChunks; ++c)
        part[c] = slots[min(c, n_chunks - 1) * SLOT + 2 + tid];   // clamped: past n_chunks never used
    if (tid < 64) {
        const bool has = tid < n_chunks;
        const float m = has ? slots[tid * SLOT] : -INFINITY;
        const float M = wave_max(m);
        const float w = has ? __builtin_amdgcn_exp2f(m - M) : 0.f;
        const float ls = wave_sum(has ? w * slots[tid * SLOT + 1] : 0.f);
        if (tid < kDecodeMaxChunks) wc[tid] = w;
        if (tid == 0) lsum = ls;
    }
    __syncthreads();
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < kDecodeMaxChunks; ++c)
        if (c < n_chunks) acc = fmaf(wc[c], part[c], acc);
    ctx[(size_t)bh * DH + tid] = to_bf16_bits(acc / lsum);
}

template <int DH>
hipError_t launch_dh(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx, int bh, int n_keys,
                     int k_rows, int vt_stride, float *partials, hipStream_t stream) {
    const float scale = 1.4426950408889634f / sqrtf((float)DH);
    const int n_chunks = decode_attention_chunks(n_keys);
    const dim3 grid(n_chunks, bh), block(kThreads);
    const hipError_t e =
        n_keys <= kSmallLimit
            ? launch_kernel(decode_attention_kernel<DH, kSmallChunk>, grid, block, stream, q, k, vt, ctx, partials,
                            n_keys, k_rows, vt_stride, scale)
            : launch_kernel(decode_attention_kernel<DH, kLargeChunk>, grid, block, stream, q, k, vt, ctx, partials,
                            n_keys, k_rows, vt_stride, scale);
    if (e != hipSuccess || n_chunks == 1) return e;
    return launch_kernel(decode_combine_kernel<DH>, dim3(bh), dim3(DH), stream, (const float *)partials, ctx,
                         n_chunks);
}

}  // namespace

int decode_attention_chunks(int n_keys) {
    const int ch = n_keys <= kSmallLimit ? kSmallChunk : kLargeChunk;
    return (n_keys + ch - 1) / ch;
}

hipError_t launch_decode_attention(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx, int batch,
                                   int n_heads, int n_keys, int head_dim, int k_rows, int vt_stride,
                                   float *partials, hipStream_t stream) {
    if (batch <= 0) return hipSuccess;
    if (n_keys <= 0 || n_keys > kMaxKeys || k_rows < n_keys || vt_stride < n_keys || vt_stride % 64 != 0 ||
        (long)batch * n_heads > 65535 || !partials)
        return hipErrorInvalidValue;
    if (head_dim == 64)
        return launch_dh<64>(q, k, vt, ctx, batch * n_heads, n_keys, k_rows, vt_stride, partials, stream);
    if (head_dim == 128)
        return launch_dh<128>(q, k, vt, ctx, batch * n_heads, n_keys, k_rows, vt_stride, partials, stream);
    return hipErrorInvalidValue;
}

}  // namespace iefwd
