// Row LayerNorm kernels (HBM-bound): one wave64 per row, the whole row held in
// registers, two-pass mean / variance with a fixed xor-butterfly reduction
// (deterministic), coalesced 16-byte accesses (8-byte when d is an odd
// multiple of 128).
//
//   layernorm : fp32 [rows, d] -> fp32 and/or bf16 [rows, d], optional {mean, rstd}
//   ln_head   : fp32 [rows, d] -> LN -> per-token head, fp32 logits [rows, n_out]
//               (the model's last LN fused with its classifier, so the final
//               hidden states never go back to HBM)
// Plus the fp32 -> bf16 cast of a post-LN model's input and the CU residency probe.
#include "kernels.h"

namespace iefwd {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kRowsPerBlock = 4;   // 4 waves, one row each

template <int VEC> struct Vec;
template <> struct Vec<2> { typedef f32x2 f; typedef uint32_t bf; };
template <> struct Vec<4> { typedef f32x4 f; typedef u32x2 bf; };

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ inline uint32_t pack2(float lo, float hi) {
    const __bf16 a = (__bf16)lo, b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// One row held by one wave: lane l owns vectors c * 64 + l (VEC floats each).
// Computes mean and rstd (two-pass, fixed butterfly order) and normalises in
// place: y = fma(gamma, (z - mean) * rstd, beta) -- the same expression the
// GEMM epilogue uses when it rebuilds a residual from the row statistics.
template <int VEC, int NC>
__device__ inline void normalize_row(typename Vec<VEC>::f (&v)[NC], const float *gamma, const float *beta,
                                     int lane, float eps, float &mean_out, float &rstd_out) {
    typedef typename Vec<VEC>::f fv;
    constexpr float inv_d = 1.0f / (float)(NC * 64 * VEC);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e) s += v[c][e];
    const float mean = wave_sum(s) * inv_d;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const float a = v[c][e] - mean;
            ss += a * a;
        }
    const float rstd = 1.0f / sqrtf(wave_sum(ss) * inv_d + eps);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int i = c * 64 + lane;
        const fv g = reinterpret_cast<const fv *>(gamma)[i];
        const fv b = reinterpret_cast<const fv *>(beta)[i];
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[c][e] = __builtin_fmaf(g[e], (v[c][e] - mean) * rstd, b[e]);
    }
    mean_out = mean;
    rstd_out = rstd;
}

template <int VEC, int NC>
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_kernel(
    const float *__restrict__ z, const float *__restrict__ gamma, const float *__restrict__ beta,
    float *__restrict__ out_f32, bf16_t *__restrict__ out_bf16, float *__restrict__ stats, int rows,
    float eps) {
    typedef typename Vec<VEC>::f fv;
    typedef typename Vec<VEC>::bf bv;
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    constexpr int D = NC * 64 * VEC;
    const fv *src = reinterpret_cast<const fv *>(z + (size_t)row * D);
    fv v[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) v[c] = src[c * 64 + lane];
    float mean, rstd;
    normalize_row<VEC, NC>(v, gamma, beta, lane, eps, mean, rstd);
    if (out_f32) {
        fv *dst = reinterpret_cast<fv *>(out_f32 + (size_t)row * D);
#pragma unroll
        for (int c = 0; c < NC; ++c) dst[c * 64 + lane] = v[c];
    }
    if (out_bf16) {
        bv *dst = reinterpret_cast<bv *>(out_bf16 + (size_t)row * D);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            if constexpr (VEC == 2) dst[c * 64 + lane] = pack2(v[c][0], v[c][1]);
            else dst[c * 64 + lane] = u32x2{pack2(v[c][0], v[c][1]), pack2(v[c][2], v[c][3])};
        }
    }
    if (stats && lane == 0) reinterpret_cast<f32x2 *>(stats)[row] = f32x2{mean, rstd};
}

template <int VEC, int NC>
__global__ __launch_bounds__(64 * kRowsPerBlock) void ln_head_kernel(
    const float *__restrict__ z, const float *__restrict__ gamma, const float *__restrict__ beta,
    const bf16_t *__restrict__ wh, const bf16_t *__restrict__ bh, float *__restrict__ logits,
    int rows, int n_out, float eps) {
    typedef typename Vec<VEC>::f fv;
    typedef typename Vec<VEC>::bf bv;
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    constexpr int D = NC * 64 * VEC;
    const fv *src = reinterpret_cast<const fv *>(z + (size_t)row * D);
    fv v[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) v[c] = src[c * 64 + lane];
    float mean, rstd;
    normalize_row<VEC, NC>(v, gamma, beta, lane, eps, mean, rstd);
    for (int o = 0; o < n_out; ++o) {
        const bv *wrow = reinterpret_cast<const bv *>(wh + (size_t)o * D);
        float part = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const bv w = wrow[c * 64 + lane];
            if constexpr (VEC == 2) {
                part += v[c][0] * __uint_as_float(w << 16) + v[c][1] * __uint_as_float(w & 0xffff0000u);
            } else {
                part += v[c][0] * __uint_as_float(w[0] << 16) + v[c][1] * __uint_as_float(w[0] & 0xffff0000u);
                part += v[c][2] * __uint_as_float(w[1] << 16) + v[c][3] * __uint_as_float(w[1] & 0xffff0000u);
            }
        }
        const float dot = wave_sum(part);
        if (lane == 0) logits[(size_t)row * n_out + o] = dot + __uint_as_float((uint32_t)bh[o] << 16);
    }
}

__global__ __launch_bounds__(256) void cast_bf16_kernel(const float *__restrict__ x, bf16_t *__restrict__ y,
                                                        size_t n4) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    const f32x4 v = reinterpret_cast<const f32x4 *>(x)[i];
    reinterpret_cast<u32x2 *>(y)[i] = u32x2{pack2(v[0], v[1]), pack2(v[2], v[3])};
}

// s_getreg immediates: register id | (offset << 6) | ((size - 1) << 11)
constexpr int kHwRegHwId = 4 | (0 << 6) | (31 << 11);    // HW_ID: wave/SIMD/CU/SH/SE fields
constexpr int kHwRegXccId = 20 | (0 << 6) | (31 << 11);  // XCC_ID

__global__ __launch_bounds__(64) void cu_probe_kernel(uint32_t *out, int n_groups) {
    if (threadIdx.x != 0 || (int)blockIdx.x >= n_groups) return;
    const uint32_t xcc = __builtin_amdgcn_s_getreg(kHwRegXccId);
    const uint32_t hw = __builtin_amdgcn_s_getreg(kHwRegHwId);
    // a little work so that the workgroups overlap in time and spread over CUs
    uint64_t t0 = __builtin_readcyclecounter();
    while (__builtin_readcyclecounter() - t0 < 20000) {}
    out[2 * blockIdx.x] = xcc;
    out[2 * blockIdx.x + 1] = hw;
}

template <int VEC, int NC>
hipError_t ln_launch(const float *z, const float *g, const float *b, float *o32, bf16_t *o16, float *stats,
                     int rows, float eps, hipStream_t s) {
    const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock), block(64 * kRowsPerBlock);
    return launch_kernel(layernorm_kernel<VEC, NC>, grid, block, s, z, g, b, o32, o16, stats, rows, eps);
}

template <int VEC, int NC>
hipError_t ln_head_launch(const float *z, const float *g, const float *b, const bf16_t *wh,
                          const bf16_t *bh, float *logits, int rows, int n_out, float eps, hipStream_t s) {
    const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock), block(64 * kRowsPerBlock);
    return launch_kernel(ln_head_kernel<VEC, NC>, grid, block, s, z, g, b, wh, bh, logits, rows, n_out, eps);
}

// d = 256 k: 16-byte vectors (k = 1..16); d = 128 (2 k + 1): 8-byte vectors
#define IEFWD_D_CASES(X) \
    X(4, 1) X(4, 2) X(4, 3) X(4, 4) X(4, 5) X(4, 6) X(4, 7) X(4, 8) X(4, 9) X(4, 10) X(4, 11) X(4, 12) \
    X(4, 13) X(4, 14) X(4, 15) X(4, 16) X(2, 1) X(2, 3) X(2, 5) X(2, 7) X(2, 9) X(2, 11) X(2, 13) X(2, 15) \
    X(2, 17) X(2, 19) X(2, 21) X(2, 23) X(2, 25) X(2, 27) X(2, 29) X(2, 31)

}  // namespace

hipError_t launch_layernorm(const float *z, const float *gamma, const float *beta, float *out_f32,
                            bf16_t *out_bf16, int rows, int d, float eps, hipStream_t stream, float *stats) {
    if (rows <= 0) return hipSuccess;
    if (d % 128 != 0) return hipErrorInvalidValue;
    const int vec = d % 256 == 0 ? 4 : 2, nc = d / (64 * vec);
#define X(V, N) \
    if (vec == V && nc == N) return ln_launch<V, N>(z, gamma, beta, out_f32, out_bf16, stats, rows, eps, stream);
    IEFWD_D_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_ln_head(const float *z, const float *gamma, const float *beta, const bf16_t *wh,
                          const bf16_t *bh, float *logits, int rows, int d, int n_out, float eps,
                          hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 128 != 0) return hipErrorInvalidValue;
    const int vec = d % 256 == 0 ? 4 : 2, nc = d / (64 * vec);
#define X(V, N) \
    if (vec == V && nc == N) return ln_head_launch<V, N>(z, gamma, beta, wh, bh, logits, rows, n_out, eps, stream);
    IEFWD_D_CASES(X)
#undef X
    return hipErrorInvalidValue;
}

hipError_t launch_cast_bf16(const float *x, bf16_t *y, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const size_t n4 = n / 4;
    const dim3 grid((unsigned)((n4 + 255) / 256)), block(256);
    return launch_kernel(cast_bf16_kernel, grid, block, stream, x, y, n4);
}

hipError_t launch_cu_probe(uint32_t *out, int n_groups, hipStream_t stream) {
    if (n_groups <= 0) return hipSuccess;
    return launch_kernel(cu_probe_kernel, dim3(n_groups), dim3(64), stream, out, n_groups);
}

}  // namespace iefwd
