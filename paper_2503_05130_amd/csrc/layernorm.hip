// Row LayerNorm kernels (HBM-bound): one wave64 per row, the whole row held in
// registers, two-pass mean / variance with a fixed xor-butterfly reduction
// (deterministic), coalesced 8-byte accesses (lane l touches floats 2l, 2l+1 of
// every 128-float chunk).
//
//   layernorm : fp32 [rows, d] -> fp32 and/or bf16 [rows, d]
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

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ inline uint32_t pack2(float lo, float hi) {
    const __bf16 a = (__bf16)lo, b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Normalises this lane's NC float2 of the row in place (affine applied).
template <int NC>
__device__ inline void normalize_row(f32x2 (&v)[NC], const float *gamma, const float *beta, int lane,
                                     float eps) {
    constexpr float inv_d = 1.0f / (float)(NC * 128);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) s += v[c][0] + v[c][1];
    const float mean = wave_sum(s) * inv_d;
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float a = v[c][0] - mean, b = v[c][1] - mean;
        ss += a * a + b * b;
    }
    const float rstd = 1.0f / sqrtf(wave_sum(ss) * inv_d + eps);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int i = c * 64 + lane;
        const f32x2 g = reinterpret_cast<const f32x2 *>(gamma)[i];
        const f32x2 b = reinterpret_cast<const f32x2 *>(beta)[i];
        v[c][0] = g[0] * ((v[c][0] - mean) * rstd) + b[0];
        v[c][1] = g[1] * ((v[c][1] - mean) * rstd) + b[1];
    }
}

template <int NC>
__global__ __launch_bounds__(64 * kRowsPerBlock) void layernorm_kernel(
    const float *__restrict__ z, const float *__restrict__ gamma, const float *__restrict__ beta,
    float *__restrict__ out_f32, bf16_t *__restrict__ out_bf16, int rows, float eps) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    constexpr int D = NC * 128;
    const f32x2 *src = reinterpret_cast<const f32x2 *>(z + (size_t)row * D);
    f32x2 v[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) v[c] = src[c * 64 + lane];
    normalize_row<NC>(v, gamma, beta, lane, eps);
    if (out_f32) {
        f32x2 *dst = reinterpret_cast<f32x2 *>(out_f32 + (size_t)row * D);
#pragma unroll
        for (int c = 0; c < NC; ++c) dst[c * 64 + lane] = v[c];
    }
    if (out_bf16) {
        uint32_t *dst = reinterpret_cast<uint32_t *>(out_bf16 + (size_t)row * D);
#pragma unroll
        for (int c = 0; c < NC; ++c) dst[c * 64 + lane] = pack2(v[c][0], v[c][1]);
    }
}

template <int NC>
__global__ __launch_bounds__(64 * kRowsPerBlock) void ln_head_kernel(
    const float *__restrict__ z, const float *__restrict__ gamma, const float *__restrict__ beta,
    const bf16_t *__restrict__ wh, const bf16_t *__restrict__ bh, float *__restrict__ logits,
    int rows, int n_out, float eps) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    constexpr int D = NC * 128;
    const f32x2 *src = reinterpret_cast<const f32x2 *>(z + (size_t)row * D);
    f32x2 v[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) v[c] = src[c * 64 + lane];
    normalize_row<NC>(v, gamma, beta, lane, eps);
    for (int o = 0; o < n_out; ++o) {
        const uint32_t *wrow = reinterpret_cast<const uint32_t *>(wh + (size_t)o * D);
        float part = 0.f;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const uint32_t w2 = wrow[c * 64 + lane];
            part += v[c][0] * __uint_as_float(w2 << 16) + v[c][1] * __uint_as_float(w2 & 0xffff0000u);
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

template <int NC>
hipError_t ln_launch(const float *z, const float *g, const float *b, float *o32, bf16_t *o16, int rows,
                     float eps, hipStream_t s) {
    const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock), block(64 * kRowsPerBlock);
    hipLaunchKernelGGL(layernorm_kernel<NC>, grid, block, 0, s, z, g, b, o32, o16, rows, eps);
    return hipGetLastError();
}

template <int NC>
hipError_t ln_head_launch(const float *z, const float *g, const float *b, const bf16_t *wh,
                          const bf16_t *bh, float *logits, int rows, int n_out, float eps, hipStream_t s) {
    const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock), block(64 * kRowsPerBlock);
    hipLaunchKernelGGL(ln_head_kernel<NC>, grid, block, 0, s, z, g, b, wh, bh, logits, rows, n_out, eps);
    return hipGetLastError();
}

// d / 128 -> template instance (d = 128 .. 4096)
#define IEFWD_NC_CASES(X) \
    X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16) \
    X(17) X(18) X(19) X(20) X(21) X(22) X(23) X(24) X(25) X(26) X(27) X(28) X(29) X(30) X(31) X(32)

}  // namespace

hipError_t launch_layernorm(const float *z, const float *gamma, const float *beta, float *out_f32,
                            bf16_t *out_bf16, int rows, int d, float eps, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 128 != 0) return hipErrorInvalidValue;
    switch (d / 128) {
#define X(n) case n: return ln_launch<n>(z, gamma, beta, out_f32, out_bf16, rows, eps, stream);
        IEFWD_NC_CASES(X)
#undef X
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_ln_head(const float *z, const float *gamma, const float *beta, const bf16_t *wh,
                          const bf16_t *bh, float *logits, int rows, int d, int n_out, float eps,
                          hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 128 != 0) return hipErrorInvalidValue;
    switch (d / 128) {
#define X(n) case n: return ln_head_launch<n>(z, gamma, beta, wh, bh, logits, rows, n_out, eps, stream);
        IEFWD_NC_CASES(X)
#undef X
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_cast_bf16(const float *x, bf16_t *y, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const size_t n4 = n / 4;
    const dim3 grid((unsigned)((n4 + 255) / 256)), block(256);
    hipLaunchKernelGGL(cast_bf16_kernel, grid, block, 0, stream, x, y, n4);
    return hipGetLastError();
}

hipError_t launch_cu_probe(uint32_t *out, int n_groups, hipStream_t stream) {
    if (n_groups <= 0) return hipSuccess;
    hipLaunchKernelGGL(cu_probe_kernel, dim3(n_groups), dim3(64), 0, stream, out, n_groups);
    return hipGetLastError();
}

}  // namespace iefwd
