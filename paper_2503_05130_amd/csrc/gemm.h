// The MFMA GEMM's interface (csrc/gemm.hip): epilogues, their operands and the
// launchers of the full-size and the decode-step (skinny) products.
#pragma once

#include "launch.h"

namespace iefwd {

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
// Requires N % 64 == 0, K % 64 == 0, M >= 1.  n_cu: the CUs the stream's mask
// enables; it may change the tile shape, never the result (every tile shape
// of a K order adds the same terms in the same order).
hipError_t launch_gemm(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                       const float *resid, void *out, int M, int N, int K,
                       const QkvDst *qkv, hipStream_t stream, const LnResid *ln = nullptr,
                       const bf16_t *aux = nullptr, int n_cu = 256);

// How launch_gemm runs a product: the K summation order (a function of the
// weight shape (N, K) alone), the order the chosen tile sums in, and the tile.
// align: the width every tile must divide (d_model for the QKV scatter, else N).
struct GemmPlan {
    bool split_order;   // K >= 2048: even / odd K tiles summed separately, then added
    bool tile_split;    // the chosen tile's order (must equal split_order)
    int bm, bn;         // output tile, tokens x features
};
GemmPlan gemm_plan(int M, int N, int K, int align, int n_cu, bool ln_residual = false);

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
// `a` is unused); that needs skinny_ln_fits(M, K).  w_packed: W's packed copy
// for packed_groups K-groups (launch_skinny_pack), read instead of w when the
// product uses that many groups for this M (bit-identical results, faster).
hipError_t launch_gemm_skinny(Epi epi, const bf16_t *a, const bf16_t *w, const bf16_t *bias,
                              const float *resid, void *out, int M, int N, int K, const QkvDst *qkv,
                              hipStream_t stream, const LnIn *ln_in = nullptr, const bf16_t *w_packed = nullptr,
                              int packed_groups = 0);
bool skinny_ln_fits(int M, int K);
// Writes dst (N * K bf16) = W [N, K] rearranged for the skinny product with
// `groups` K-groups: each 1 KB block holds one workgroup's fragment of one
// 32-wide K step in lane order.  Needs N % (16 / groups) == 0 and
// K % (32 * groups) == 0.
hipError_t launch_skinny_pack(const bf16_t *w, bf16_t *dst, int N, int K, int groups, hipStream_t stream);
// K-groups per MFMA the skinny product uses for this shape (1, 2 or 4), with
// or without the LayerNorm prologue; its summation order depends on K and
// this number.
int skinny_groups(int M, int N, int K, bool ln);

}  // namespace iefwd
