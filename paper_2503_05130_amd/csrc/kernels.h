// Launchers of the forward-pass kernels (gfx950).  Host-callable; every
// launcher validates nothing beyond what its kernel's indexing needs -- shape
// checks live in the callers (executor and test entry points).
#pragma once

#include "gemm.h"
#include "launch.h"

namespace iefwd {

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
// combines them.  partials: at least B * H * decode_attention_chunks(n_keys)
// * (dh + 2) floats of scratch, every one of them written before it is read
// (nothing needs clearing); launches sharing it must not overlap.
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
