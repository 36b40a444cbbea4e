// Training-step kernels for gfx950: what a post-LN encoder's backward pass and
// optimiser need beyond the forward kernels and the GEMM.
//
//   transpose          bf16 [R, C] -> [C, R] through 64 x 64 LDS tiles (the
//                      GEMM contracts over its operands' contiguous dimension,
//                      so weight gradients, which contract over tokens, read
//                      transposed activations); several in one launch; on
//                      request also the per-64-row column sums of the source
//                      (the bias gradients' first stage)
//   colsum             per row block: column sums (fp32 or bf16 input), fixed
//                      order; the last stages of several sums in one launch
//   gelu               u = GELU(v), bf16 -> bf16
//   ln_backward        dz = rstd (g - mean(g) - x^ mean(g x^)), g = dy gamma,
//                      one wave per row, fp32; writes fp32 and bf16
//   ln_param_partials  per 256-row chunk: sum dy x^ and sum dy per column
//   ln_backward_params ln_backward with the parameter partials of 16-row
//                      blocks (d <= 1024: one pass over dy and z)
//   head_loss          per token: the last LayerNorm, logits = X Wh^T + bh,
//                      softmax cross-entropy, dlogits = (p - onehot) / N,
//                      dX = dlogits Wh
//   head_partials      per 256-row chunk: sum dlogits^T X (the head's gradient)
//   attention_backward per (batch, head), S <= 128, MFMA: P recomputed from Q
//                      and K, dS = P (dP - D), D = rowsum(dO O); dQ, dK, dV
//   adamw              one pass over every parameter (fp32 master, moments),
//                      writing the forward's bf16 (or fp32) copy
// Every reduction runs in a fixed order, so a training step is deterministic.
#include "gelu.h"
#include "kernels.h"

namespace iefwd {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline float bf(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline uint16_t to_bf(float f) {
    __bf16 b = (__bf16)f;   // round to nearest even
    return __builtin_bit_cast(uint16_t, b);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

// ------------------------------------------------------------------ transpose
constexpr int kTile = 64;

// One 64 x 64 tile of a bf16 [R, C] -> [C, R] transpose: rows r0.., columns c0.. of src.
// With colsum non-null, also colsum[(r0 / 64) * C + c0 + c] = sum over the tile's
// rows of column c: thread (c, q) adds rows 16 q .. 16 q + 15 in order, then the
// four partial sums are added in q order.
__device__ inline void transpose_tile(const uint16_t *__restrict__ src, uint16_t *__restrict__ dst, int R, int C,
                                      int r0, int c0, uint16_t (&tile)[kTile][kTile + 2], float *__restrict__ colsum,
                                      float (&red)[4][kTile]) {
    const int tid = threadIdx.x;
    // in: rows r0 + tid / 8 (+ 32), 8 columns each (16 bytes)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int r = tid / 8 + 32 * h, c = (tid % 8) * 8;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(src + (size_t)(r0 + r) * C + c0 + c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            tile[r][c + 2 * e] = (uint16_t)(v[e] & 0xffffu);
            tile[r][c + 2 * e + 1] = (uint16_t)(v[e] >> 16);
        }
    }
    __syncthreads();
    // out: rows c0 + tid / 8 (+ 32) of dst, 8 source rows each
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int cc = tid / 8 + 32 * h, rr = (tid % 8) * 8;
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (uint32_t)tile[rr + 2 * e][cc] | ((uint32_t)tile[rr + 2 * e + 1][cc] << 16);
        *reinterpret_cast<u32x4 *>(dst + (size_t)(c0 + cc) * R + r0 + rr) = v;
    }
    if (colsum) {   // uniform over the workgroup
        const int c = tid & 63, q = tid >> 6;
        float sum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += bf(tile[16 * q + r][c]);
        red[q][c] = sum;
        __syncthreads();
        if (q == 0) colsum[(size_t)(r0 / kTile) * C + c0 + c] = red[0][c] + red[1][c] + red[2][c] + red[3][c];
    }
}

__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t *__restrict__ src, uint16_t *__restrict__ dst,
                                                        int R, int C) {
    __shared__ uint16_t tile[kTile][kTile + 2];
    __shared__ float red[4][kTile];
    transpose_tile(src, dst, R, C, blockIdx.y * kTile, blockIdx.x * kTile, tile, nullptr, red);
}

// Several transposes in one launch: workgroup b takes tile b - first[j] of the
// job j with first[j] <= b < first[j + 1] (tiles numbered row-major per job).
struct TransposeBatch {
    TransposeJob job[kMaxTransposeJobs];
    int32_t first[kMaxTransposeJobs + 1];
    int32_t n;
};

__global__ __launch_bounds__(256) void transpose_jobs_kernel(TransposeBatch b) {
    __shared__ uint16_t tile[kTile][kTile + 2];
    __shared__ float red[4][kTile];
    int j = 0;
    while (j + 1 < b.n && (int)blockIdx.x >= b.first[j + 1]) ++j;
    const int t = (int)blockIdx.x - b.first[j], tiles_c = b.job[j].cols / kTile;
    transpose_tile(reinterpret_cast<const uint16_t *>(b.job[j].src), reinterpret_cast<uint16_t *>(b.job[j].dst),
                   b.job[j].rows, b.job[j].cols, (t / tiles_c) * kTile, (t % tiles_c) * kTile, tile, b.job[j].colsum,
                   red);
}

// ------------------------------------------------------------------ GELU
__global__ __launch_bounds__(256) void gelu_kernel(const uint16_t *__restrict__ v, uint16_t *__restrict__ u,
                                                   size_t n8) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n8) return;
    const u32x4 x = reinterpret_cast<const u32x4 *>(v)[i];
    u32x4 y;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float lo = gelu(__uint_as_float(x[e] << 16)), hi = gelu(__uint_as_float(x[e] & 0xffff0000u));
        y[e] = (uint32_t)to_bf(lo) | ((uint32_t)to_bf(hi) << 16);
    }
    reinterpret_cast<u32x4 *>(u)[i] = y;
}

// ------------------------------------------------------------------ LayerNorm backward
constexpr int kRowsPerBlock = 4;   // one wave per row

// Two passes over the row (the second re-reads dy and z from the cache):
// sums of g and g x^, then dz.  x^ = (z - mean) rstd with the forward's
// statistics.  d % 4 == 0.
__global__ __launch_bounds__(64 * kRowsPerBlock) void ln_backward_kernel(
    const float *__restrict__ dy, const float *__restrict__ z, const float *__restrict__ stats,
    const float *__restrict__ gamma, float *__restrict__ dz, uint16_t *__restrict__ dzb, int rows, int d) {
    const int lane = threadIdx.x & 63, row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    const float mean = stats[2 * (size_t)row], rstd = stats[2 * (size_t)row + 1];
    const f32x4 *dyr = reinterpret_cast<const f32x4 *>(dy + (size_t)row * d);
    const f32x4 *zr = reinterpret_cast<const f32x4 *>(z + (size_t)row * d);
    const f32x4 *g4 = reinterpret_cast<const f32x4 *>(gamma);
    const int nv = d / 4;
    float sg = 0.f, sgx = 0.f;
    for (int i = lane; i < nv; i += 64) {
        const f32x4 a = dyr[i], zz = zr[i], g = g4[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float gg = a[e] * g[e], xh = (zz[e] - mean) * rstd;
            sg += gg;
            sgx += gg * xh;
        }
    }
    const float inv_d = 1.0f / (float)d;
    const float mg = wave_sum(sg) * inv_d, mgx = wave_sum(sgx) * inv_d;
    for (int i = lane; i < nv; i += 64) {
        const f32x4 a = dyr[i], zz = zr[i], g = g4[i];
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float xh = (zz[e] - mean) * rstd;
            o[e] = rstd * (a[e] * g[e] - mg - xh * mgx);
        }
        if (dz) reinterpret_cast<f32x4 *>(dz + (size_t)row * d)[i] = o;
        reinterpret_cast<u32x2 *>(dzb + (size_t)row * d)[i] =
            u32x2{(uint32_t)to_bf(o[0]) | ((uint32_t)to_bf(o[1]) << 16), (uint32_t)to_bf(o[2]) | ((uint32_t)to_bf(o[3]) << 16)};
    }
}

// LayerNorm backward fused with the first stage of its parameter gradients,
// for d <= 256 NV: a workgroup of 4 waves takes 4 RPW consecutive rows (wave w
// rows w RPW .. w RPW + RPW - 1, each as in ln_backward_kernel) and keeps, per
// lane, the running sums of dy x^ and dy over its rows for its columns; the
// four waves' sums are added in wave order into the block's partial row.
template <int NV, int RPW>
__global__ __launch_bounds__(256) void ln_backward_params_kernel(
    const float *__restrict__ dy, const float *__restrict__ z, const float *__restrict__ stats,
    const float *__restrict__ gamma, float *__restrict__ dz, uint16_t *__restrict__ dzb, float *__restrict__ part_g,
    float *__restrict__ part_b, int rows, int d) {
    __shared__ float red[2][4][256 * NV];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nv = d / 4, blk = blockIdx.x;
    const f32x4 *g4 = reinterpret_cast<const f32x4 *>(gamma);
    f32x4 gm[NV], pg[NV], pb[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int i = v * 64 + lane;
        gm[v] = i < nv ? g4[i] : f32x4{0.f, 0.f, 0.f, 0.f};
        pg[v] = pb[v] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const float inv_d = 1.0f / (float)d;
    for (int k = 0; k < RPW; ++k) {
        const int row = (blk * 4 + wave) * RPW + k;
        if (row >= rows) break;   // wave-uniform
        const float mean = stats[2 * (size_t)row], rstd = stats[2 * (size_t)row + 1];
        const f32x4 *dyr = reinterpret_cast<const f32x4 *>(dy + (size_t)row * d);
        const f32x4 *zr = reinterpret_cast<const f32x4 *>(z + (size_t)row * d);
        f32x4 a[NV], xh[NV];
        float sg = 0.f, sgx = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int i = v * 64 + lane;
            a[v] = xh[v] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (i < nv) {
                a[v] = dyr[i];
                const f32x4 zz = zr[i];
#pragma unroll
                for (int e = 0; e < 4; ++e) xh[v][e] = (zz[e] - mean) * rstd;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float gg = a[v][e] * gm[v][e];
                sg += gg;
                sgx += gg * xh[v][e];
            }
        }
        const float mg = wave_sum(sg) * inv_d, mgx = wave_sum(sgx) * inv_d;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int i = v * 64 + lane;
            if (i >= nv) continue;
            f32x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                o[e] = rstd * (a[v][e] * gm[v][e] - mg - xh[v][e] * mgx);
                pg[v][e] += a[v][e] * xh[v][e];
                pb[v][e] += a[v][e];
            }
            if (dz) reinterpret_cast<f32x4 *>(dz + (size_t)row * d)[i] = o;
            reinterpret_cast<u32x2 *>(dzb + (size_t)row * d)[i] =
                u32x2{(uint32_t)to_bf(o[0]) | ((uint32_t)to_bf(o[1]) << 16), (uint32_t)to_bf(o[2]) | ((uint32_t)to_bf(o[3]) << 16)};
        }
    }
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            red[0][wave][4 * (v * 64 + lane) + e] = pg[v][e];
            red[1][wave][4 * (v * 64 + lane) + e] = pb[v][e];
        }
    __syncthreads();
    for (int f = threadIdx.x; f < d; f += 256) {
        part_g[(size_t)blk * d + f] = red[0][0][f] + red[0][1][f] + red[0][2][f] + red[0][3][f];
        part_b[(size_t)blk * d + f] = red[1][0][f] + red[1][1][f] + red[1][2][f] + red[1][3][f];
    }
}
constexpr int kLnbRowsPerWave = 4;

// ------------------------------------------------------------------ column sums
// A workgroup sums 64 columns over one chunk of kColRows rows: thread (column
// c, lane g of 4) adds rows g, g + 4, ... of the chunk in order, then lane 0
// adds the 4 lanes' sums in order.  Fixed order, so the sums are deterministic.
constexpr int kColRows = 256;   // rows per partial
constexpr int kColLanes = 4;

__device__ inline float lane_total(float v, int c, int g, float (&red)[kColLanes][64]) {
    red[g][c] = v;
    __syncthreads();
    return red[0][c] + red[1][c] + red[2][c] + red[3][c];
}

// partial_g[b][f] = sum over rows of chunk b of dy x^, partial_b[b][f] = sum dy
__global__ __launch_bounds__(256) void ln_param_partials_kernel(
    const float *__restrict__ dy, const float *__restrict__ z, const float *__restrict__ stats,
    float *__restrict__ part_g, float *__restrict__ part_b, int rows, int d) {
    __shared__ float red[kColLanes][64];
    const int c = threadIdx.x & 63, g = threadIdx.x >> 6, f = blockIdx.x * 64 + c, b = blockIdx.y;
    float sg = 0.f, sb = 0.f;
    if (f < d) {
        const int r1 = min(rows, (b + 1) * kColRows);
#pragma unroll 4
        for (int r = b * kColRows + g; r < r1; r += kColLanes) {
            const float a = dy[(size_t)r * d + f];
            sg += a * ((z[(size_t)r * d + f] - stats[2 * (size_t)r]) * stats[2 * (size_t)r + 1]);
            sb += a;
        }
    }
    const float tg = lane_total(sg, c, g, red);
    __syncthreads();
    const float tb = lane_total(sb, c, g, red);
    if (g == 0 && f < d) {
        part_g[(size_t)b * d + f] = tg;
        part_b[(size_t)b * d + f] = tb;
    }
}

template <typename T>
__device__ inline float load_as_f32(const T *p, size_t i);
template <>
__device__ inline float load_as_f32<float>(const float *p, size_t i) { return p[i]; }
template <>
__device__ inline float load_as_f32<uint16_t>(const uint16_t *p, size_t i) { return bf(p[i]); }

// One workgroup's column block: dst[b * n + f] = sum of src rows b * rb ..
// min(rows, b * rb + rb) - 1 of column f, f = 64 cb .. 64 cb + 63
template <typename T>
__device__ inline void colsum_block(const T *__restrict__ src, float *__restrict__ dst, int rows, int n, int rb,
                                    int cb, int b, float (&red)[kColLanes][64]) {
    const int c = threadIdx.x & 63, g = threadIdx.x >> 6, f = cb * 64 + c;
    float s = 0.f;
    if (f < n) {
        const int r1 = min(rows, (b + 1) * rb);
#pragma unroll 4
        for (int r = b * rb + g; r < r1; r += kColLanes) s += load_as_f32(src, (size_t)r * n + f);
    }
    const float t = lane_total(s, c, g, red);
    if (g == 0 && f < n) dst[(size_t)b * n + f] = t;
}

template <typename T>
__global__ __launch_bounds__(256) void colsum_kernel(const T *__restrict__ src, float *__restrict__ dst, int rows,
                                                     int n, int rb) {
    __shared__ float red[kColLanes][64];
    colsum_block(src, dst, rows, n, rb, blockIdx.x, blockIdx.y, red);
}

// Several whole-column sums in one launch (the last stage of a layer's sums:
// a few hundred partial rows each).  Workgroup b takes 32 columns of job j
// (first[j] <= b < first[j + 1]); thread (column c, lane g of 8) adds rows g,
// g + 8, ... in order, then lane 0 adds the 8 lanes' sums in order.
constexpr int kFinCols = 32, kFinLanes = 8;

struct ColsumBatch {
    ColsumJob job[kMaxColsumJobs];
    int32_t first[kMaxColsumJobs + 1];
    int32_t n;
};

__global__ __launch_bounds__(256) void colsum_jobs_kernel(ColsumBatch b) {
    __shared__ float red[kFinLanes][kFinCols];
    int j = 0;
    while (j + 1 < b.n && (int)blockIdx.x >= b.first[j + 1]) ++j;
    const float *__restrict__ src = b.job[j].src;
    const int rows = b.job[j].rows, n = b.job[j].n;
    const int c = threadIdx.x % kFinCols, g = threadIdx.x / kFinCols;
    const int f = ((int)blockIdx.x - b.first[j]) * kFinCols + c;
    float sum = 0.f;
    if (f < n) {
#pragma unroll 4
        for (int r = g; r < rows; r += kFinLanes) sum += src[(size_t)r * n + f];
    }
    red[g][c] = sum;
    __syncthreads();
    if (g == 0 && f < n) {
        float t = red[0][c];
#pragma unroll
        for (int k = 1; k < kFinLanes; ++k) t += red[k][c];
        b.job[j].dst[f] = t;
    }
}

// ------------------------------------------------------------------ head + loss
// One wave per token.  The last LayerNorm (two-pass statistics, the forward
// LayerNorm kernel's expression), logits = X Wh^T + bh, softmax cross-entropy
// against the label, dlogits = (p - onehot) * inv_n, dX = dlogits Wh.
// Writes X (fp32), the statistics, logits, per-token loss, dlogits and dX.
// d % 4 == 0, n_out <= 16.
__global__ __launch_bounds__(64 * kRowsPerBlock) void head_loss_kernel(
    const float *__restrict__ z, const float *__restrict__ gamma, const float *__restrict__ beta,
    const uint16_t *__restrict__ wh, const uint16_t *__restrict__ bh, const int32_t *__restrict__ labels,
    float *__restrict__ xl, float *__restrict__ stats, float *__restrict__ logits, float *__restrict__ loss_t,
    float *__restrict__ dlogits, float *__restrict__ dx, int rows, int d, int n_out, float eps, float inv_n) {
    const int lane = threadIdx.x & 63, row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int nv = d / 4;
    const f32x4 *zr = reinterpret_cast<const f32x4 *>(z + (size_t)row * d);
    float s = 0.f;
    for (int i = lane; i < nv; i += 64) {
        const f32x4 a = zr[i];
        s += a[0] + a[1] + a[2] + a[3];
    }
    const float inv_d = 1.0f / (float)d;
    const float mean = wave_sum(s) * inv_d;
    float ss = 0.f;
    for (int i = lane; i < nv; i += 64) {
        const f32x4 a = zr[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float c = a[e] - mean;
            ss += c * c;
        }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(ss) * inv_d + eps);
    float acc[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[c] = 0.f;
    for (int i = lane; i < nv; i += 64) {
        const f32x4 a = zr[i], g = reinterpret_cast<const f32x4 *>(gamma)[i], b = reinterpret_cast<const f32x4 *>(beta)[i];
        f32x4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __builtin_fmaf(g[e], (a[e] - mean) * rstd, b[e]);
        reinterpret_cast<f32x4 *>(xl + (size_t)row * d)[i] = x;
#pragma unroll
        for (int c = 0; c < 16; ++c)
            if (c < n_out) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(wh + (size_t)c * d + 4 * i);
                acc[c] += x[0] * __uint_as_float(w[0] << 16) + x[1] * __uint_as_float(w[0] & 0xffff0000u) +
                          x[2] * __uint_as_float(w[1] << 16) + x[3] * __uint_as_float(w[1] & 0xffff0000u);
            }
    }
    float lg[16], mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < 16; ++c)
        if (c < n_out) {
            lg[c] = wave_sum(acc[c]) + bf(bh[c]);
            mx = fmaxf(mx, lg[c]);
        }
    float se = 0.f;
#pragma unroll
    for (int c = 0; c < 16; ++c)
        if (c < n_out) se += __expf(lg[c] - mx);
    const float lse = mx + __logf(se);
    const int label = labels[row];
    float dl[16];
#pragma unroll
    for (int c = 0; c < 16; ++c)
        if (c < n_out) dl[c] = (__expf(lg[c] - lse) - (c == label ? 1.0f : 0.0f)) * inv_n;
    if (lane < n_out) {
        float l = 0.f, g = 0.f;
#pragma unroll
        for (int c = 0; c < 16; ++c)
            if (c == lane) {
                l = lg[c];
                g = dl[c];
            }
        logits[(size_t)row * n_out + lane] = l;
        dlogits[(size_t)row * n_out + lane] = g;
    }
    if (lane == 0) {
        float ll = 0.f;
#pragma unroll
        for (int c = 0; c < 16; ++c)
            if (c == label) ll = lg[c];
        loss_t[row] = lse - ll;
        stats[2 * (size_t)row] = mean;
        stats[2 * (size_t)row + 1] = rstd;
    }
    for (int i = lane; i < nv; i += 64) {
        f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 16; ++c)
            if (c < n_out) {
                const u32x2 w = *reinterpret_cast<const u32x2 *>(wh + (size_t)c * d + 4 * i);
                o[0] += dl[c] * __uint_as_float(w[0] << 16);
                o[1] += dl[c] * __uint_as_float(w[0] & 0xffff0000u);
                o[2] += dl[c] * __uint_as_float(w[1] << 16);
                o[3] += dl[c] * __uint_as_float(w[1] & 0xffff0000u);
            }
        reinterpret_cast<f32x4 *>(dx + (size_t)row * d)[i] = o;
    }
}

// part[b][k * d + f] = sum over rows of chunk b of dlogits[r][k] * xl[r][f]
__global__ __launch_bounds__(256) void head_partials_kernel(const float *__restrict__ dlogits,
                                                            const float *__restrict__ xl, float *__restrict__ part,
                                                            int rows, int d, int n_out) {
    __shared__ float red[kColLanes][64];
    const int c = threadIdx.x & 63, g = threadIdx.x >> 6, idx = blockIdx.x * 64 + c, b = blockIdx.y;
    float s = 0.f;
    if (idx < n_out * d) {
        const int k = idx / d, f = idx - k * d;
        const int r1 = min(rows, (b + 1) * kColRows);
#pragma unroll 4
        for (int r = b * kColRows + g; r < r1; r += kColLanes) s += dlogits[(size_t)r * n_out + k] * xl[(size_t)r * d + f];
    }
    const float t = lane_total(s, c, g, red);
    if (g == 0 && idx < n_out * d) part[(size_t)b * n_out * d + idx] = t;
}

// ------------------------------------------------------------------ attention backward
// One workgroup (4 waves) per (batch, head); S <= 128 keys, head dim 64, all
// five products on v_mfma_f32_32x32x16_bf16.  (32x32x16 operands: lane l holds
// A[l % 32][8 (l / 32) .. +8] and B[8 (l / 32) .. +8][l % 32]; accumulator
// entry r of lane l is C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].)
//   load     Q, K, V, dO of the head into LDS in row layout ([token][c]);
//            D_i = sum_c dO[i][c] O[i][c].  Rows past S are zero.
//   phase 1  wave w, queries 32 w .. 32 w + 31: S^T = K Q^T and dP^T = V dO^T
//            (keys as rows, so a lane holds 64 of its query's 128 keys, its
//            partner lane l ^ 32 the rest); softmax over keys in registers
//            (causal: keys j <= i), dS = P (dP - D_i).  P^T and dS^T ([key]
//            [query]) and dS ([query][key]) go to a per-head scratch in global
//            memory (L2-resident), the layouts phase 2 reads as A operands.
//   relayout Q, K and dO move from the row copies (through registers) to
//            transposed copies ([c][token]) in the same LDS, which phase 2
//            reads as B operands.  Only one layout is ever resident, so a
//            workgroup takes 74 KB of LDS and two share a CU.
//   phase 2  wave w: dV = P^T dO and dK = dS^T Q for keys 32 w .. 32 w + 31,
//            dQ = dS K for queries 32 w .. 32 w + 31 (dQ and dK times
//            1 / sqrt(dh)).
// fp32 accumulation and softmax; P and dS are rounded to bf16 for phase 2.
constexpr int kAbSeq = 128, kAbDh = 64;
constexpr int kAbLd = kAbDh + 8, kAbLdT = kAbSeq + 8;   // LDS row strides (bf16)
constexpr size_t kAbScratch = 3 * (size_t)kAbSeq * kAbSeq;   // bf16 elements per head

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline bf16x8 ld8(const uint16_t *p) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p)); }

__global__ __launch_bounds__(256) void attention_backward_kernel(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K, const uint16_t *__restrict__ Vt,
    const uint16_t *__restrict__ ctx, const uint16_t *__restrict__ dctx, uint16_t *__restrict__ dqkv,
    uint16_t *__restrict__ scratch, int n_heads, int S, int vt_stride, int causal, float scale) {
    // row copies for phase 1; the transposed copies of phase 2 reuse the same space
    static_assert(3 * kAbDh * kAbLdT <= 4 * kAbSeq * kAbLd, "transposed copies fit the row copies' space");
    __shared__ __attribute__((aligned(16))) uint16_t lds[4 * kAbSeq * kAbLd];
    __shared__ float sD[kAbSeq];
    uint16_t *sQ = lds, *sK = sQ + kAbSeq * kAbLd, *sV = sK + kAbSeq * kAbLd, *sdO = sV + kAbSeq * kAbLd;
    uint16_t *sQt = lds, *sKt = sQt + kAbDh * kAbLdT, *sdOt = sKt + kAbDh * kAbLdT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5, col = lane & 31;
    const int bh = blockIdx.x, b = bh / n_heads, h = bh - b * n_heads;
    const int d = n_heads * kAbDh;
    const size_t tok0 = (size_t)b * S;
    const uint16_t *Qh = Q + (size_t)bh * S * kAbDh, *Kh = K + (size_t)bh * S * kAbDh;
    const uint16_t *Vh = Vt + (size_t)bh * kAbDh * vt_stride;
    uint16_t *Pt = scratch + (size_t)bh * kAbScratch, *dSt = Pt + kAbSeq * kAbSeq, *dS = dSt + kAbSeq * kAbSeq;

    // ---- load: 8-element vectors, row i = v / 8, columns c0 .. c0 + 7
    const u32x4 zero = {0u, 0u, 0u, 0u};
    for (int v = tid; v < kAbSeq * kAbDh / 8; v += 256) {
        const int i = v / 8, c0 = (v % 8) * 8;
        const bool in = i < S;
        const u32x4 q = in ? *reinterpret_cast<const u32x4 *>(Qh + (size_t)i * kAbDh + c0) : zero;
        const u32x4 k = in ? *reinterpret_cast<const u32x4 *>(Kh + (size_t)i * kAbDh + c0) : zero;
        const u32x4 g = in ? *reinterpret_cast<const u32x4 *>(dctx + (tok0 + i) * d + h * kAbDh + c0) : zero;
        const u32x4 o = in ? *reinterpret_cast<const u32x4 *>(ctx + (tok0 + i) * d + h * kAbDh + c0) : zero;
        *reinterpret_cast<u32x4 *>(sQ + i * kAbLd + c0) = q;
        *reinterpret_cast<u32x4 *>(sK + i * kAbLd + c0) = k;
        *reinterpret_cast<u32x4 *>(sdO + i * kAbLd + c0) = g;
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            dot += __uint_as_float(g[e] << 16) * __uint_as_float(o[e] << 16) +
                   __uint_as_float(g[e] & 0xffff0000u) * __uint_as_float(o[e] & 0xffff0000u);
        // the 8 vectors of row i are 8 consecutive lanes
#pragma unroll
        for (int m = 4; m >= 1; m >>= 1) dot += __shfl_xor(dot, m);
        if (v % 8 == 0) sD[i] = dot;
    }
    // V from V^T [c][j]: vector v = 8 keys j0 .. j0 + 7 of column c; keys past S are zero
    for (int v = tid; v < kAbDh * kAbSeq / 8; v += 256) {
        const int c = v / (kAbSeq / 8), j0 = (v % (kAbSeq / 8)) * 8;
        u32x4 x = j0 < S ? *reinterpret_cast<const u32x4 *>(Vh + (size_t)c * vt_stride + j0) : zero;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint16_t val = j0 + e < S ? (uint16_t)(x[e / 2] >> (16 * (e % 2))) : (uint16_t)0;
            sV[(j0 + e) * kAbLd + c] = val;
        }
    }
    __syncthreads();

    // ---- phase 1: queries of this wave against all keys
    const int iq = 32 * wave + col;          // this lane's query
    f32x16 st[4], dpt[4];
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) st[jb][r] = dpt[jb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < kAbDh / 16; ++ks) {
            const int kc = 16 * ks + 8 * half;
            st[jb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(sK + (32 * jb + col) * kAbLd + kc),
                                                             ld8(sQ + iq * kAbLd + kc), st[jb], 0, 0, 0);
            dpt[jb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(sV + (32 * jb + col) * kAbLd + kc),
                                                              ld8(sdO + iq * kAbLd + kc), dpt[jb], 0, 0, 0);
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int j = 32 * jb + 8 * (r / 4) + 4 * half + r % 4;
            const bool ok = iq < S && j < S && (!causal || j <= iq);
            st[jb][r] = ok ? st[jb][r] * scale : -INFINITY;
            mx = fmaxf(mx, st[jb][r]);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float l = 0.f;
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float p = st[jb][r] == -INFINITY ? 0.f : __expf(st[jb][r] - mx);
            st[jb][r] = p;
            l += p;
        }
    l += __shfl_xor(l, 32);
    const float inv_l = iq < S ? 1.0f / l : 0.f;
    const float Di = sD[iq];
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            uint16_t dsv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 4 * q4 + e, j = 32 * jb + 8 * q4 + 4 * half + e;
                const float p = st[jb][r] * inv_l, ds = p * (dpt[jb][r] - Di);
                Pt[j * kAbSeq + iq] = to_bf(p);
                dsv[e] = to_bf(ds);
                dSt[j * kAbSeq + iq] = dsv[e];
            }
            *reinterpret_cast<u32x2 *>(dS + iq * kAbSeq + 32 * jb + 8 * q4 + 4 * half) =
                u32x2{(uint32_t)dsv[0] | ((uint32_t)dsv[1] << 16), (uint32_t)dsv[2] | ((uint32_t)dsv[3] << 16)};
        }

    // ---- relayout: Q, K, dO rows -> registers -> transposed copies over the same LDS
    constexpr int kVecs = kAbSeq * kAbDh / 8 / 256;   // 8-element row vectors per thread and matrix
    u32x4 rq[kVecs], rk[kVecs], rg[kVecs];
#pragma unroll
    for (int u = 0; u < kVecs; ++u) {
        const int v = tid + 256 * u, i = v / 8, c0 = (v % 8) * 8;
        rq[u] = *reinterpret_cast<const u32x4 *>(sQ + i * kAbLd + c0);
        rk[u] = *reinterpret_cast<const u32x4 *>(sK + i * kAbLd + c0);
        rg[u] = *reinterpret_cast<const u32x4 *>(sdO + i * kAbLd + c0);
    }
    __syncthreads();   // every wave is done with the row copies
#pragma unroll
    for (int u = 0; u < kVecs; ++u) {
        const int v = tid + 256 * u, i = v / 8, c0 = (v % 8) * 8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sQt[(c0 + 2 * e) * kAbLdT + i] = (uint16_t)(rq[u][e] & 0xffffu);
            sQt[(c0 + 2 * e + 1) * kAbLdT + i] = (uint16_t)(rq[u][e] >> 16);
            sKt[(c0 + 2 * e) * kAbLdT + i] = (uint16_t)(rk[u][e] & 0xffffu);
            sKt[(c0 + 2 * e + 1) * kAbLdT + i] = (uint16_t)(rk[u][e] >> 16);
            sdOt[(c0 + 2 * e) * kAbLdT + i] = (uint16_t)(rg[u][e] & 0xffffu);
            sdOt[(c0 + 2 * e + 1) * kAbLdT + i] = (uint16_t)(rg[u][e] >> 16);
        }
    }
    __syncthreads();   // the transposed copies and the scratch are complete (workgroup scope)

    // ---- phase 2: keys 32 w .. 32 w + 31 (dV, dK) and queries 32 w .. 32 w + 31 (dQ)
    f32x16 dv[2], dk[2], dq[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) dv[cb][r] = dk[cb][r] = dq[cb][r] = 0.f;
    const int row = 32 * wave + col;
#pragma unroll
    for (int ks = 0; ks < kAbSeq / 16; ++ks) {
        const int kc = 16 * ks + 8 * half;
        const bf16x8 a_p = ld8(Pt + row * kAbSeq + kc), a_dst = ld8(dSt + row * kAbSeq + kc);
        const bf16x8 a_ds = ld8(dS + row * kAbSeq + kc);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int c = 32 * cb + col;
            dv[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_p, ld8(sdOt + c * kAbLdT + kc), dv[cb], 0, 0, 0);
            dk[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_dst, ld8(sQt + c * kAbLdT + kc), dk[cb], 0, 0, 0);
            dq[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_ds, ld8(sKt + c * kAbLdT + kc), dq[cb], 0, 0, 0);
        }
    }
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int t = 32 * wave + 8 * (r / 4) + 4 * half + r % 4, c = 32 * cb + col;
            if (t >= S) continue;
            uint16_t *o = dqkv + (tok0 + t) * 3 * d + h * kAbDh + c;
            o[0] = to_bf(dq[cb][r] * scale);
            o[d] = to_bf(dk[cb][r] * scale);
            o[2 * d] = to_bf(dv[cb][r]);
        }
}

// ------------------------------------------------------------------ AdamW
// One thread per 4 consecutive parameters (16-byte loads and stores; the
// scalar form for a segment's last, partial group); block b covers parameters
// of segment blk_seg[b] only (segments start at multiples of kAdamBlock
// elements, and every out pointer is 16-byte aligned).
constexpr int kAdamBlock = 1024;

struct AdamOne {
    float w, m, v;
};

__device__ inline AdamOne adam_one(float w, float g, float m, float v, float decay, const AdamStep &st) {
    const float mm = st.beta1 * m + (1.0f - st.beta1) * g;
    const float vv = st.beta2 * v + (1.0f - st.beta2) * g * g;
    const float upd = (mm * st.c1) / (sqrtf(vv * st.c2) + st.eps);
    return {w * decay - st.lr * upd, mm, vv};
}

__global__ __launch_bounds__(256) void adamw_kernel(float *__restrict__ w, const float *__restrict__ g,
                                                    float *__restrict__ m, float *__restrict__ v,
                                                    const AdamSegment *__restrict__ segs,
                                                    const uint32_t *__restrict__ blk_seg, AdamStep st) {
    const AdamSegment sg = segs[blk_seg[blockIdx.x]];
    const size_t base = (size_t)blockIdx.x * kAdamBlock;
    const size_t i0 = base + threadIdx.x * 4, end = sg.offset + sg.count;
    if (i0 >= end) return;
    const float decay = sg.decay ? 1.0f - st.lr * st.weight_decay : 1.0f;
    const size_t k0 = i0 - sg.offset;
    if (i0 + 4 <= end) {
        const f32x4 gg = *reinterpret_cast<const f32x4 *>(g + i0);
        const f32x4 mm = *reinterpret_cast<const f32x4 *>(m + i0);
        const f32x4 vv = *reinterpret_cast<const f32x4 *>(v + i0);
        const f32x4 ww = *reinterpret_cast<const f32x4 *>(w + i0);
        f32x4 nw, nm, nv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const AdamOne r = adam_one(ww[e], gg[e], mm[e], vv[e], decay, st);
            nw[e] = r.w;
            nm[e] = r.m;
            nv[e] = r.v;
        }
        *reinterpret_cast<f32x4 *>(m + i0) = nm;
        *reinterpret_cast<f32x4 *>(v + i0) = nv;
        *reinterpret_cast<f32x4 *>(w + i0) = nw;
        if (sg.out_bf16)
            *reinterpret_cast<u32x2 *>(static_cast<uint16_t *>(sg.out) + k0) =
                u32x2{(uint32_t)to_bf(nw[0]) | ((uint32_t)to_bf(nw[1]) << 16),
                      (uint32_t)to_bf(nw[2]) | ((uint32_t)to_bf(nw[3]) << 16)};
        else
            *reinterpret_cast<f32x4 *>(static_cast<float *>(sg.out) + k0) = nw;
        return;
    }
    for (size_t i = i0; i < end; ++i) {
        const AdamOne r = adam_one(w[i], g[i], m[i], v[i], decay, st);
        m[i] = r.m;
        v[i] = r.v;
        w[i] = r.w;
        if (sg.out_bf16) static_cast<uint16_t *>(sg.out)[i - sg.offset] = to_bf(r.w);
        else static_cast<float *>(sg.out)[i - sg.offset] = r.w;
    }
}

__global__ __launch_bounds__(256) void bf16_to_f32_kernel(const uint16_t *__restrict__ src, float *__restrict__ dst,
                                                          size_t n) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = bf(src[i]);
}

}  // namespace

hipError_t launch_transpose_bf16(const bf16_t *src, bf16_t *dst, int R, int C, hipStream_t stream) {
    if (R <= 0 || C <= 0) return hipSuccess;
    if (R % kTile || C % kTile) return hipErrorInvalidValue;
    return launch_kernel(transpose_kernel, dim3(C / kTile, R / kTile), dim3(256), stream, src, dst, R, C);
}

hipError_t launch_transposes(const TransposeJob *jobs, int n_jobs, hipStream_t stream) {
    if (n_jobs <= 0) return hipSuccess;
    if (n_jobs > kMaxTransposeJobs) return hipErrorInvalidValue;
    TransposeBatch b{};
    b.n = n_jobs;
    long tiles = 0;
    for (int j = 0; j < n_jobs; ++j) {
        const TransposeJob &jb = jobs[j];
        if (jb.rows <= 0 || jb.cols <= 0 || jb.rows % kTile || jb.cols % kTile) return hipErrorInvalidValue;
        b.job[j] = jb;
        b.first[j] = (int32_t)tiles;
        tiles += (long)(jb.rows / kTile) * (jb.cols / kTile);
        if (tiles > 0x7fffffffL) return hipErrorInvalidValue;
    }
    b.first[n_jobs] = (int32_t)tiles;
    return launch_kernel(transpose_jobs_kernel, dim3((unsigned)tiles), dim3(256), stream, b);
}

hipError_t launch_colsums(const ColsumJob *jobs, int n_jobs, hipStream_t stream) {
    if (n_jobs <= 0) return hipSuccess;
    if (n_jobs > kMaxColsumJobs) return hipErrorInvalidValue;
    ColsumBatch b{};
    b.n = n_jobs;
    int blocks = 0;
    for (int j = 0; j < n_jobs; ++j) {
        if (jobs[j].rows <= 0 || jobs[j].n <= 0) return hipErrorInvalidValue;
        b.job[j] = jobs[j];
        b.first[j] = blocks;
        blocks += (jobs[j].n + kFinCols - 1) / kFinCols;
    }
    b.first[n_jobs] = blocks;
    return launch_kernel(colsum_jobs_kernel, dim3(blocks), dim3(kFinCols * kFinLanes), stream, b);
}

hipError_t launch_gelu(const bf16_t *v, bf16_t *u, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (n % 8) return hipErrorInvalidValue;
    const size_t n8 = n / 8;
    return launch_kernel(gelu_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), stream, v, u, n8);
}

hipError_t launch_ln_backward(const float *dy, const float *z, const float *stats, const float *gamma, float *dz,
                              bf16_t *dzb, int rows, int d, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 4) return hipErrorInvalidValue;
    return launch_kernel(ln_backward_kernel, dim3((rows + kRowsPerBlock - 1) / kRowsPerBlock),
                         dim3(64 * kRowsPerBlock), stream, dy, z, stats, gamma, dz, dzb, rows, d);
}

int colsum_partials(int rows) { return (rows + kColRows - 1) / kColRows; }

int ln_backward_partials(int rows, int d) {
    return d <= 1024 ? (rows + 4 * kLnbRowsPerWave - 1) / (4 * kLnbRowsPerWave) : colsum_partials(rows);
}

hipError_t launch_ln_backward_params(const float *dy, const float *z, const float *stats, const float *gamma,
                                     float *dz, bf16_t *dzb, float *part_g, float *part_b, int rows, int d,
                                     hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 4) return hipErrorInvalidValue;
    if (d > 1024) {   // registers hold at most 16 columns per lane: the two-kernel form
        const hipError_t e = launch_ln_backward(dy, z, stats, gamma, dz, dzb, rows, d, stream);
        if (e != hipSuccess) return e;
        return launch_ln_param_partials(dy, z, stats, part_g, part_b, rows, d, stream);
    }
    const dim3 grid(ln_backward_partials(rows, d)), block(256);
    const int nv = d / 4;
    if (nv <= 64)
        return launch_kernel(ln_backward_params_kernel<1, kLnbRowsPerWave>, grid, block, stream, dy, z, stats, gamma,
                             dz, dzb, part_g, part_b, rows, d);
    if (nv <= 128)
        return launch_kernel(ln_backward_params_kernel<2, kLnbRowsPerWave>, grid, block, stream, dy, z, stats, gamma,
                             dz, dzb, part_g, part_b, rows, d);
    if (nv <= 192)
        return launch_kernel(ln_backward_params_kernel<3, kLnbRowsPerWave>, grid, block, stream, dy, z, stats, gamma,
                             dz, dzb, part_g, part_b, rows, d);
    return launch_kernel(ln_backward_params_kernel<4, kLnbRowsPerWave>, grid, block, stream, dy, z, stats, gamma, dz,
                         dzb, part_g, part_b, rows, d);
}

hipError_t launch_ln_param_partials(const float *dy, const float *z, const float *stats, float *part_g,
                                    float *part_b, int rows, int d, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    return launch_kernel(ln_param_partials_kernel, dim3((d + 63) / 64, colsum_partials(rows)), dim3(256), stream,
                         dy, z, stats, part_g, part_b, rows, d);
}

hipError_t launch_colsum(const void *src, bool src_bf16, float *dst, int rows, int n, int rows_per_part,
                         hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    const dim3 grid((n + 63) / 64, (rows + rows_per_part - 1) / rows_per_part);
    if (src_bf16)
        return launch_kernel(colsum_kernel<uint16_t>, grid, dim3(256), stream, static_cast<const uint16_t *>(src), dst,
                             rows, n, rows_per_part);
    return launch_kernel(colsum_kernel<float>, grid, dim3(256), stream, static_cast<const float *>(src), dst, rows, n,
                         rows_per_part);
}

hipError_t launch_head_loss(const float *z, const float *gamma, const float *beta, const bf16_t *wh,
                            const bf16_t *bh, const int32_t *labels, float *xl, float *stats, float *logits,
                            float *loss_t, float *dlogits, float *dx, int rows, int d, int n_out, float eps,
                            float inv_n, hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    if (d % 4 || n_out < 1 || n_out > 16) return hipErrorInvalidValue;
    return launch_kernel(head_loss_kernel, dim3((rows + kRowsPerBlock - 1) / kRowsPerBlock), dim3(64 * kRowsPerBlock),
                         stream, z, gamma, beta, wh, bh, labels, xl, stats, logits, loss_t, dlogits, dx, rows, d,
                         n_out, eps, inv_n);
}

hipError_t launch_head_partials(const float *dlogits, const float *xl, float *part, int rows, int d, int n_out,
                                hipStream_t stream) {
    if (rows <= 0) return hipSuccess;
    return launch_kernel(head_partials_kernel, dim3((n_out * d + 63) / 64, colsum_partials(rows)), dim3(256), stream,
                         dlogits, xl, part, rows, d, n_out);
}

size_t attention_backward_scratch(int batch, int n_heads) { return (size_t)batch * n_heads * kAbScratch; }

hipError_t launch_attention_backward(const bf16_t *q, const bf16_t *k, const bf16_t *vt, const bf16_t *ctx,
                                     const bf16_t *dctx, bf16_t *dqkv, bf16_t *scratch, int batch, int n_heads,
                                     int seq, int head_dim, int vt_stride, bool causal, hipStream_t stream) {
    if (batch <= 0) return hipSuccess;
    if (seq < 1 || seq > kAbSeq || vt_stride < seq || vt_stride % 8 || head_dim != kAbDh || !scratch)
        return hipErrorInvalidValue;
    return launch_kernel(attention_backward_kernel, dim3(batch * n_heads), dim3(256), stream, q, k, vt, ctx, dctx, dqkv,
                         scratch, n_heads, seq, vt_stride, causal ? 1 : 0, 1.0f / sqrtf((float)head_dim));
}

hipError_t launch_adamw(float *w, const float *g, float *m, float *v, const AdamSegment *segs,
                        const uint32_t *blk_seg, int n_blocks, const AdamStep &st, hipStream_t stream) {
    if (n_blocks <= 0) return hipSuccess;
    return launch_kernel(adamw_kernel, dim3(n_blocks), dim3(kAdamBlock / 4), stream, w, g, m, v, segs, blk_seg, st);
}

int adamw_block() { return kAdamBlock; }

hipError_t launch_bf16_to_f32(const bf16_t *src, float *dst, size_t n, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    return launch_kernel(bf16_to_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), stream, src, dst, n);
}

}  // namespace iefwd
