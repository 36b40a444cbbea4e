// Launchers of the forward-pass kernels (gfx950).  Host-callable; every
// launcher validates nothing beyond what its kernel's indexing needs -- shape
// checks live in the callers (executor and test entry points).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace iefwd {

// Kernel-only timing: when a pair of events is armed on this host thread, the
// next kernel launch records its own dispatch start and end into them (the
// timestamps of the kernel itself, not of markers around it) and disarms.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
// Events armed by the caller for the next launches on this thread: the first
// kernel records `start` as it begins, and every kernel records `stop` as it
// ends, so for an operation of several kernels the pair spans all of them.
LaunchEvents &armed_launch_events();
// Kernels launched by this thread so far.
uint64_t &launch_count();

template <typename F, typename... Args>
hipError_t launch_kernel(F kernel, dim3 grid, dim3 block, hipStream_t stream, Args... args) {
    LaunchEvents &ev = armed_launch_events();
    if (ev.stop) {
        hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
        ev.start = nullptr;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
    }
    ++launch_count();
    return hipGetLastError();
}

using bf16_t = uint16_t;   // bf16 storage: the upper half of an fp32 bit pattern

enum class Epi : int {
    BiasBf16 = 0,       // out bf16 = acc + b
    BiasGeluBf16 = 1,   // out bf16 = GELU(acc + b)
    BiasResidF32 = 2,   // out f32  = resid + acc + b
    Qkv = 3,            // acc + b scattered to Q, K [B,H,S,dh] and V^T [B,H,dh,S_pad]
    BiasLnResidF32 = 4, // out f32  = LN(z) + acc + b, LN(z) rebuilt from z and its row stats
    F32 = 5,            // out f32  = acc                      (weight gradients)
    GeluBwdBf16 = 6,    // out bf16 = acc * GELU'(aux), aux bf16 [M, N] (the GELU's input)
};

// Row statistics a LayerNorm kernel leaves for a later consumer: the residual
// LN(z)[t, f] = gamma[f] * ((z[t, f] - mean[t]) * rstd[t]) + beta[f] is rebuilt
// from them with exactly the LayerNorm kernel's arithmetic.
struct LnResid {
    const float *z;       // [M, N] fp32 pre-normalisation rows
    const float *stats;   // [M, 2] fp32 {mean, rstd}
    const float *gamma;   // [N]
    const float *beta;    // [N]
};

// Destination of the QKV epilogue.
// Where the QKV epilogue puts each token's Q, K and V.  Token t of a launch is
// position pos0 + t % seq of sequence t / seq.  Q goes to the per-launch
// buffer [B, H, seq, dh]; K and V^T go to buffers that may be a KV cache:
// K [B, H, k_rows, dh] at row pos0 + t % seq, V^T [B, H, dh, vt_stride] at
// column pos0 + t % seq.  A prefill without a cache has pos0 = 0,
// k_rows = seq, vt_stride = S rounded up to a multiple of 64.
struct QkvDst {
    bf16_t *q, *k, *vt;
    int seq;        // tokens per sequence in this launch
    int pos0;       // position of the launch's first token of each sequence
    int k_rows;     // rows of K per (batch, head)
    int vt_stride;  // row stride of V^T (a multiple of 64)
    int n_heads;
    int head_dim;
    int d_model;
};

// S rounded up to the attention kernel's 64-key chunk (the row stride of V^T).
inline int attn_seq_pad(int seq) { return (seq + 63) / 64 * 64; }

// out = epi(A W^T + b).  A bf16 [M,K], W bf16 [N,K], bias bf16 [N].
// Requires N % 64 == 0, K % 64 == 0, M >= 1.
hipError_t launch_gemm(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                       const float *resid, void *out, int M, int N, int K,
                       const QkvDst *qkv, hipStream_t stream, const LnResid *ln = nullptr,
                       const bf16_t *aux = nullptr);

// Activations given as LayerNorm(z): z fp32 [M, K] rows, gamma / beta fp32 [K].
struct LnIn {
    const float *z;
    const float *gamma;
    const float *beta;
    float eps;
};

// The same product for M <= 16 rows (a decode step), bound by reading W once:
// N % 16 == 0, K % 32 == 0; every epilogue but BiasLnResidF32.  Its K
// summation order differs from launch_gemm's (the two agree within rounding).
// With ln_in the activations are LayerNorm(z), normalised in the kernel (then
// `a` is unused); that needs skinny_ln_fits(M, K).
hipError_t launch_gemm_skinny(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                              const float *resid, void *out, int M, int N, int K, const QkvDst *qkv,
                              hipStream_t stream, const LnIn *ln_in = nullptr);
bool skinny_ln_fits(int M, int K);
// K-groups per MFMA the skinny product uses for this shape (1, 2 or 4), with
// or without the LayerNorm prologue; its summation order depends on K and
// this number.
int skinny_groups(int M, int N, int K, bool ln);

// ctx bf16 [B, S, H*dh] from Q, K [B,H,S,dh] and V^T [B,H,dh,S_pad].
// k_rows: rows of K per (batch, head) (0: seq); vt_stride: row stride of V^T
// (0: seq rounded up to 64), so that K and V^T may live in a longer KV cache.
hipError_t launch_attention(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx,
                            int batch, int n_heads, int seq, int head_dim, bool causal,
                            hipStream_t stream, int k_rows = 0, int vt_stride = 0);

// Attention of one new query per (batch, head) over keys 0 .. n_keys - 1 of a
// KV cache: q bf16 [B, H, dh], K [B, H, k_rows, dh], V^T [B, H, dh, vt_stride];
// ctx bf16 [B, H * dh].  fp32 scores, softmax and sums.  n_keys <= 8192.
// The keys are split into decode_attention_chunks(n_keys) <= kDecodeMaxChunks
// chunks, one workgroup each; with more than one chunk a second kernel
// combines them.  partials: at least B * H * kDecodeMaxChunks * (dh + 2)
// floats of scratch; launches sharing it must not overlap.
constexpr int kDecodeMaxChunks = 32;
int decode_attention_chunks(int n_keys);
hipError_t launch_decode_attention(const bf16_t *q, const bf16_t *k, const bf16_t *vt, bf16_t *ctx,
                                   int batch, int n_heads, int n_keys, int head_dim, int k_rows,
                                   int vt_stride, float *partials, hipStream_t stream);

// ---- training step (csrc/train.hip) ----
// bf16 [R, C] -> [C, R]; R % 64 == 0, C % 64 == 0.
hipError_t launch_transpose_bf16(const bf16_t *src, bf16_t *dst, int R, int C, hipStream_t stream);
// Up to kMaxTransposeJobs such transposes (bf16 src [rows, cols] -> dst [cols, rows]) in one launch.
// With colsum non-null the job also writes the column sums of each 64-row block
// of src: colsum[b * cols + c] = sum of src[64 b .. 64 b + 63][c] (fp32, a fixed order).
struct TransposeJob {
    const bf16_t *src;
    bf16_t *dst;
    int32_t rows, cols;
    float *colsum = nullptr;
};
constexpr int kMaxTransposeJobs = 48;
hipError_t launch_transposes(const TransposeJob *jobs, int n_jobs, hipStream_t stream);
// u = GELU(v) elementwise, bf16; n % 8 == 0.
hipError_t launch_gelu(const bf16_t *v, bf16_t *u, size_t n, hipStream_t stream);
// LayerNorm backward per row: dz = rstd (g - mean(g) - x^ mean(g x^)), g = dy gamma,
// x^ = (z - mean) rstd with the forward's {mean, rstd}.  dz (fp32, may be null)
// and dzb (bf16) [rows, d]; d % 4 == 0.
hipError_t launch_ln_backward(const float *dy, const float *z, const float *stats, const float *gamma, float *dz,
                              bf16_t *dzb, int rows, int d, hipStream_t stream);
// Column-sum partials over chunks of 256 rows: colsum_partials(rows) of them.
int colsum_partials(int rows);
// part_g[b][f] = sum_r dy x^, part_b[b][f] = sum_r dy over the rows of chunk b.
hipError_t launch_ln_param_partials(const float *dy, const float *z, const float *stats, float *part_g,
                                    float *part_b, int rows, int d, hipStream_t stream);
// launch_ln_backward and the parameter partials together: part_g / part_b get
// ln_backward_partials(rows, d) rows (row blocks of 16 rows for d <= 1024,
// one pass over dy and z; else the 256-row chunks of launch_ln_param_partials).
int ln_backward_partials(int rows, int d);
hipError_t launch_ln_backward_params(const float *dy, const float *z, const float *stats, const float *gamma,
                                     float *dz, bf16_t *dzb, float *part_g, float *part_b, int rows, int d,
                                     hipStream_t stream);
// dst[b][f] = sum of src[r][f] over rows b * rows_per_part .. (b + 1) * rows_per_part - 1, in row order.
hipError_t launch_colsum(const void *src, bool src_bf16, float *dst, int rows, int n, int rows_per_part,
                         hipStream_t stream);
// Up to kMaxColsumJobs whole-column sums of fp32 [rows, n] matrices in one launch:
// dst[f] = sum of src[r][f] over all rows, in a fixed order (8 interleaved row
// lanes, each in row order, then the lanes in order).
struct ColsumJob {
    const float *src;
    float *dst;
    int32_t rows, n;
};
constexpr int kMaxColsumJobs = 16;
hipError_t launch_colsums(const ColsumJob *jobs, int n_jobs, hipStream_t stream);
// Per token: the last LayerNorm of z (two-pass statistics), logits = X Wh^T + bh,
// softmax cross-entropy against labels, dlogits = (p - onehot) * inv_n, dX = dlogits Wh.
// Writes xl = X (fp32 [rows, d]), stats, logits and dlogits [rows, n_out],
// loss_t [rows] (the token's loss) and dx [rows, d].  n_out <= 16.
hipError_t launch_head_loss(const float *z, const float *gamma, const float *beta, const bf16_t *wh,
                            const bf16_t *bh, const int32_t *labels, float *xl, float *stats, float *logits,
                            float *loss_t, float *dlogits, float *dx, int rows, int d, int n_out, float eps,
                            float inv_n, hipStream_t stream);
// part[b][c * d + f] = sum over chunk b's rows of dlogits[r][c] xl[r][f].
hipError_t launch_head_partials(const float *dlogits, const float *xl, float *part, int rows, int d, int n_out,
                                hipStream_t stream);
// Attention backward for seq <= 128, head_dim 64: from Q, K [B,H,S,dh], V^T
// [B,H,dh,vt_stride], the forward's context and its gradient (bf16 [B*S, H*dh])
// to dQ | dK | dV as bf16 [B*S, 3 H dh] (the QKV product's column order).
// scratch: attention_backward_scratch(batch, n_heads) bf16 elements.
size_t attention_backward_scratch(int batch, int n_heads);
hipError_t launch_attention_backward(const bf16_t *q, const bf16_t *k, const bf16_t *vt, const bf16_t *ctx,
                                     const bf16_t *dctx, bf16_t *dqkv, bf16_t *scratch, int batch, int n_heads,
                                     int seq, int head_dim, int vt_stride, bool causal, hipStream_t stream);

// One parameter tensor of the flat AdamW state: elements offset .. offset +
// count - 1 (offset a multiple of adamw_block()); after the update the new
// value is also written to out[k] (bf16 when out_bf16, else fp32).
struct AdamSegment {
    size_t offset;
    size_t count;
    void *out;
    int32_t out_bf16;
    int32_t decay;
};
// Hyper-parameters of one step; c1 = 1 / (1 - beta1^t), c2 = 1 / (1 - beta2^t).
struct AdamStep {
    float lr, beta1, beta2, eps, weight_decay, c1, c2;
};
int adamw_block();
hipError_t launch_adamw(float *w, const float *g, float *m, float *v, const AdamSegment *segs,
                        const uint32_t *blk_seg, int n_blocks, const AdamStep &st, hipStream_t stream);
hipError_t launch_bf16_to_f32(const bf16_t *src, float *dst, size_t n, hipStream_t stream);

// Row LayerNorm, d % 128 == 0, d <= 4096.  out_f32 / out_bf16 / stats may be
// null; stats receives {mean, rstd} per row.
hipError_t launch_layernorm(const float *z, const float *gamma, const float *beta,
                            float *out_f32, bf16_t *out_bf16, int rows, int d, float eps,
                            hipStream_t stream, float *stats = nullptr);

// LayerNorm + per-token head: logits [rows, n_out] = LN(z) Wh^T + bh, Wh bf16 [n_out, d].
hipError_t launch_ln_head(const float *z, const float *gamma, const float *beta,
                          const bf16_t *wh, const bf16_t *bh, float *logits, int rows, int d,
                          int n_out, float eps, hipStream_t stream);

// bf16 copy of an fp32 array (round to nearest even); n % 4 == 0.
hipError_t launch_cast_bf16(const float *x, bf16_t *y, size_t n, hipStream_t stream);

// One 64-thread workgroup per entry: out[2g] = XCC id, out[2g+1] = HW_ID register.
hipError_t launch_cu_probe(uint32_t *out, int n_groups, hipStream_t stream);

}  // namespace iefwd
