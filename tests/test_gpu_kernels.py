"""Per-kernel parity on the GPU: each HIP kernel, called through the C ABI,
against the oracle's definition of the same step on the same bf16/fp32 inputs.

Bounds are derived from the arithmetic: bf16 x bf16 products are exact in
fp32, so a K-term fp32 accumulation is within gamma_K * sum|a||w| of the exact
sum (Higham, Accuracy and Stability of Numerical Algorithms, Sec. 3.1), plus
half an ulp of the output format (bf16: at most 2^-8 relative)."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
from oracle import forward as F
from tests.gpu_util import DEV, bf16_round, f64, sync, to_dev

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24     # fp32 unit roundoff
UBF = 2.0 ** -8      # bf16 unit roundoff: 8 significant bits, round to nearest


def gemm_inputs(M, N, K, seed, scale_w=0.05):
    rng = np.random.default_rng(seed)
    a = bf16_round(rng.standard_normal((M, K)))
    w_logical = bf16_round(rng.standard_normal((K, N)) * scale_w)      # [in, out]
    bias = bf16_round(rng.standard_normal(N) * 0.1)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    return a, w_logical, bias, resid


def gemm_bound(a64, w64, K):
    return (K + 16) * U32 * (np.abs(a64) @ np.abs(w64)) + 1e-7


@pytest.mark.parametrize("M,N,K", [
    (64, 384, 128),      # one-layer encoder QKV shape
    (1, 64, 64),         # single row
    (37, 192, 128),      # ragged M, 64 x 64 tiles
    (130, 320, 192),     # ragged M over several tiles
    (1000, 768, 768),    # 64 x 64 tiles (most tiles), ragged M
    (512, 3072, 768),    # 64 x 96 tiles, 4 waves
    (4096, 3072, 256),   # 128 x 192 tiles, 8 waves
    (4125, 2496, 128),   # 128 x 192 tiles, ragged M
    (4096, 1024, 256),   # 128 x 128 tiles, 8 waves
    (4096, 768, 768),    # 128 x 96 tiles, 8 waves
    (2000, 1024, 512),   # 64 x 128 tiles, ragged M
    (300, 1024, 1024),   # 64 x 64 tiles, ragged M
    (256, 768, 3072),    # long K: split (even/odd) K order, 64 x 96
    (130, 512, 2048),    # split order, small product: 32 x 64, ragged M
    (768, 768, 4096),    # split order, small product: 32 x 64 (an out-projection weight gradient)
    (1000, 1024, 2048),  # split order, small product: 32 x 64, ragged M
    (2000, 768, 2048),   # split order, 64 x 96, ragged M (just past the small-product limit)
    (2048, 2048, 2048),  # split order, 128 x 128
    (4096, 768, 3072),   # split order, 64 x 96 (the BERT-base FFN-down product)
    (4133, 768, 2048),   # split order, 64 x 96, ragged M
])
@pytest.mark.parametrize("epi", [ie.EPI_BIAS_BF16, ie.EPI_BIAS_GELU_BF16, ie.EPI_BIAS_RESID_F32])
def test_gemm_epilogues(M, N, K, epi):
    print(f"gemm M={M} N={N} K={K} epi={epi}", flush=True)
    a, w, bias, resid = gemm_inputs(M, N, K, seed=M * 7 + N + K + epi)
    a_d, w_d, b_d = to_dev(a), to_dev(w.t()), to_dev(bias)       # W stored [N, K]
    r_d = torch.from_numpy(resid).to(DEV)
    out = torch.empty((M, N), dtype=torch.float32 if epi == ie.EPI_BIAS_RESID_F32 else torch.bfloat16,
                      device=DEV)
    ie.test_gemm(epi, a_d, w_d, b_d, r_d if epi == ie.EPI_BIAS_RESID_F32 else None, out, M, N, K)
    sync()
    a64, w64, b64 = f64(a), f64(w), f64(bias)
    pre = F.linear(a64, w64, b64)
    bound = gemm_bound(a64, w64, K)
    got = f64(out)
    if epi == ie.EPI_BIAS_BF16:
        ref = pre
        tol = bound + UBF * np.abs(ref) * 1.01
    elif epi == ie.EPI_BIAS_GELU_BF16:
        ref = F.gelu(pre)
        # |GELU'| <= 1.13; erff error ~1e-7 relative
        tol = 1.13 * bound + UBF * np.abs(ref) * 1.01 + 1e-6 * np.abs(pre) + 1e-7
    else:
        ref = pre + resid.astype(np.float64)
        tol = bound + 2 * U32 * (np.abs(ref) + np.abs(resid)) + 1e-7
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got))
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert np.all(err <= tol), f"max excess at {worst}: err {err[worst]} tol {tol[worst]}"


@pytest.mark.parametrize("M,N,K", [
    (512, 768, 768),      # 64 x 64 tiles throughout
    (4096, 3072, 768),    # 128 x 192 tiles (8 waves) for the full batch, 64 x 64 / 64 x 96 for the slices
    (4096, 1024, 4096),   # split K order: 128 x 128 for the full batch, 32 x 64 for the slices
    (4096, 768, 3072),    # split K order: 64 x 96 for the full batch (the BERT-base FFN-down
                          # product), 32 x 64 for the slices
    (2048, 768, 4096),    # split K order: 64 x 96 for the full batch, 32 x 64 for the slices
])
def test_gemm_batch_invariance(M, N, K):
    # rows computed in a large batch equal the same rows computed alone, bit for
    # bit, even when the two launches pick different tile shapes
    a, w, bias, _ = gemm_inputs(M, N, K, seed=3)
    a_d, w_d, b_d = to_dev(a), to_dev(w.t()), to_dev(bias)
    full = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    ie.test_gemm(ie.EPI_BIAS_BF16, a_d, w_d, b_d, None, full, M, N, K)
    for lo, hi in [(0, 1), (100, 137), (384, 512)]:
        part = torch.empty((hi - lo, N), dtype=torch.bfloat16, device=DEV)
        ie.test_gemm(ie.EPI_BIAS_BF16, a_d[lo:hi].contiguous(), w_d, b_d, None, part, hi - lo, N, K)
        sync()
        assert torch.equal(part.view(torch.int16), full[lo:hi].view(torch.int16))


@pytest.mark.parametrize("B,S,d,H", [
    (2, 32, 128, 2), (3, 37, 256, 2), (2, 128, 768, 12), (1, 70, 1024, 8),
    (33, 125, 768, 12),   # 128 x 192 tiles, S not a multiple of 8 (V^T element stores), ragged M
    (32, 128, 768, 12),   # 128 x 192 tiles, V^T 16-byte stores
    (8, 512, 1024, 16),   # d = 1024: tile widths must divide d (128 x 128)
    (2, 1024, 2048, 16),  # K = 2048: split K order with the scatter (dh 128)
])
def test_qkv_scatter(B, S, d, H):
    print(f"qkv B={B} S={S} d={d} H={H}", flush=True)
    dh = d // H
    M = B * S
    a, w, bias, _ = gemm_inputs(M, 3 * d, d, seed=B + S + d)
    spad = (S + 63) // 64 * 64
    q = torch.empty((B, H, S, dh), dtype=torch.bfloat16, device=DEV)
    k = torch.empty_like(q)
    vt = torch.zeros((B, H, dh, spad), dtype=torch.bfloat16, device=DEV)
    ie.test_gemm_qkv(to_dev(a), to_dev(w.t()), to_dev(bias), q, k, vt, B, S, d, H)
    sync()
    a64, w64 = f64(a), f64(w)
    ref = F.linear(a64, w64, f64(bias)).reshape(B, S, 3, H, dh)
    bound = gemm_bound(a64, w64, d).reshape(B, S, 3, H, dh)
    want = [ref[:, :, i].transpose(0, 2, 1, 3) for i in range(3)]        # [B, H, S, dh]
    tols = [bound[:, :, i].transpose(0, 2, 1, 3) + UBF * 1.01 * np.abs(want[i]) + 1e-7 for i in range(3)]
    got = [f64(q), f64(k), f64(vt)[..., :S].transpose(0, 1, 3, 2)]
    for g, r, t in zip(got, want, tols):
        assert np.all(np.abs(g - r) <= t)


def attn_inputs(B, H, S, dh, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    q = bf16_round(rng.standard_normal((B, H, S, dh)) * scale)
    k = bf16_round(rng.standard_normal((B, H, S, dh)) * scale)
    v = bf16_round(rng.standard_normal((B, H, S, dh)))
    return q, k, v


@pytest.mark.parametrize("B,H,S,dh,causal", [
    (2, 2, 32, 64, False),
    (1, 3, 128, 64, False),
    (2, 2, 37, 64, False),     # ragged key / query tail
    (2, 2, 37, 64, True),
    (1, 1, 1, 64, False),      # single token
    (1, 1, 1, 128, True),
    (1, 2, 200, 128, True),
    (2, 4, 512, 64, True),     # decoder prefill, several workgroups per head
    (1, 2, 1024, 128, True),
    (1, 2, 300, 128, False),
    (24, 12, 230, 64, True),   # 576 heads x 128-query groups: 4-wave workgroups
    (6, 16, 700, 128, False),
])
@pytest.mark.parametrize("scale", [0.5, 2.0])
def test_attention(B, H, S, dh, causal, scale):
    print(f"attention B={B} H={H} S={S} dh={dh} causal={causal} scale={scale}", flush=True)
    q, k, v = attn_inputs(B, H, S, dh, seed=S + dh + B, scale=scale)
    spad = (S + 63) // 64 * 64
    vt = torch.full((B, H, dh, spad), float("nan"), dtype=torch.bfloat16)   # padding must be ignored
    vt[..., :S] = v.transpose(2, 3)
    ctx = torch.empty((B, S, H * dh), dtype=torch.bfloat16, device=DEV)
    ie.test_attention(to_dev(q), to_dev(k), to_dev(vt), ctx, B, H, S, dh, causal)
    sync()
    ref = F.attention_context(f64(q), f64(k), f64(v), causal)               # [B, H, S, dh]
    ref = ref.transpose(0, 2, 1, 3).reshape(B, S, H * dh)
    got = f64(ctx)
    vmax = np.abs(f64(v)).max()
    # P rounded to bf16 (2^-9 relative each) + bf16 output + fp32 scores/exp
    tol = 2.5 * UBF * vmax + UBF * 1.01 * np.abs(ref) + 1e-4 * vmax
    assert np.all(np.isfinite(got))
    assert np.all(np.abs(got - ref) <= tol), float(np.max(np.abs(got - ref) - tol))


@pytest.mark.parametrize("dh,causal", [(64, False), (64, True), (128, True)])
def test_attention_batch_invariant(dh, causal):
    """A head's context does not depend on how many other heads share the
    launch: a large batch (128-query workgroups) and a one-sequence launch
    (64-query workgroups) give the same bits."""
    B, H, S = 40, 13, 200
    print(f"attention batch invariance dh={dh} causal={causal}", flush=True)
    q, k, v = attn_inputs(B, H, S, dh, seed=dh + 7)
    vt = torch.zeros((B, H, dh, 256), dtype=torch.bfloat16)
    vt[..., :S] = v.transpose(2, 3)
    full = torch.empty((B, S, H * dh), dtype=torch.bfloat16, device=DEV)
    ie.test_attention(to_dev(q), to_dev(k), to_dev(vt), full, B, H, S, dh, causal)
    for b in (0, 17, B - 1):
        one = torch.empty((1, S, H * dh), dtype=torch.bfloat16, device=DEV)
        ie.test_attention(to_dev(q[b:b + 1]), to_dev(k[b:b + 1]), to_dev(vt[b:b + 1]), one, 1, H, S, dh, causal)
        sync()
        assert torch.equal(one[0].view(torch.int16), full[b].view(torch.int16)), b


def test_attention_uniform_closed_form():
    # all-zero Q and K: every visible key gets the same weight -> mean / prefix mean of V
    B, H, S, dh = 1, 2, 96, 64
    q = torch.zeros((B, H, S, dh), dtype=torch.bfloat16)
    _, _, v = attn_inputs(B, H, S, dh, seed=5)
    spad = 128
    for causal in (False, True):
        vt = torch.zeros((B, H, dh, spad), dtype=torch.bfloat16)
        vt[..., :S] = v.transpose(2, 3)
        ctx = torch.empty((B, S, H * dh), dtype=torch.bfloat16, device=DEV)
        ie.test_attention(to_dev(q), to_dev(q), to_dev(vt), ctx, B, H, S, dh, causal)
        sync()
        v64 = f64(v)
        if causal:
            want = np.cumsum(v64, axis=2) / np.arange(1, S + 1)[None, None, :, None]
        else:
            want = np.broadcast_to(v64.mean(axis=2, keepdims=True), v64.shape)
        want = want.transpose(0, 2, 1, 3).reshape(B, S, H * dh)
        tol = 2.5 * UBF * np.abs(v64).max() + UBF * np.abs(want)
        assert np.all(np.abs(f64(ctx) - want) <= tol)
        assert spad == vt.shape[-1]


@pytest.mark.parametrize("rows,d", [(1, 128), (37, 768), (300, 1024), (64, 2048), (5, 4096)])
def test_layernorm(rows, d):
    print(f"layernorm rows={rows} d={d}", flush=True)
    rng = np.random.default_rng(rows + d)
    z = (rng.standard_normal((rows, d)) * 3 + 2).astype(np.float32)
    g = (1 + 0.3 * rng.standard_normal(d)).astype(np.float32)
    b = (0.3 * rng.standard_normal(d)).astype(np.float32)
    o32 = torch.empty((rows, d), dtype=torch.float32, device=DEV)
    o16 = torch.empty((rows, d), dtype=torch.bfloat16, device=DEV)
    zd, gd, bd = (torch.from_numpy(t).to(DEV) for t in (z, g, b))
    ie.test_layernorm(zd, gd, bd, o32, o16, rows, d, 1e-5)
    sync()
    ref = F.layer_norm(z.astype(np.float64), g.astype(np.float64), b.astype(np.float64), 1e-5)
    xhat = np.abs(ref - b) / np.maximum(np.abs(g), 1e-30)
    tol32 = 1e-5 * (np.abs(g) * (xhat + 1) + np.abs(b)) + 1e-6
    assert np.all(np.abs(f64(o32) - ref) <= tol32)
    assert np.all(np.abs(f64(o16) - ref) <= tol32 + UBF * 1.01 * np.abs(ref))
    # the bf16 output is exactly the RNE rounding of the fp32 output
    assert torch.equal(o32.to(torch.bfloat16).view(torch.int16), o16.view(torch.int16))


@pytest.mark.parametrize("rows,d,n_out", [(64, 128, 2), (130, 768, 2), (17, 1024, 5), (8, 2048, 16)])
def test_ln_head(rows, d, n_out):
    print(f"ln_head rows={rows} d={d} n_out={n_out}", flush=True)
    rng = np.random.default_rng(rows * d + n_out)
    z = (rng.standard_normal((rows, d)) * 2 - 1).astype(np.float32)
    g = (1 + 0.2 * rng.standard_normal(d)).astype(np.float32)
    b = (0.2 * rng.standard_normal(d)).astype(np.float32)
    wh = bf16_round(rng.standard_normal((d, n_out)) * 0.05)     # logical [in, out]
    bh = bf16_round(rng.standard_normal(n_out) * 0.1)
    logits = torch.empty((rows, n_out), dtype=torch.float32, device=DEV)
    zd, gd, bd = (torch.from_numpy(t).to(DEV) for t in (z, g, b))
    ie.test_ln_head(zd, gd, bd, to_dev(wh.t()), to_dev(bh), logits, rows, d, n_out, 1e-5)
    sync()
    y = F.layer_norm(z.astype(np.float64), g.astype(np.float64), b.astype(np.float64), 1e-5)
    ref = F.linear(y, f64(wh), f64(bh))
    tol = (d + 8) * U32 * (np.abs(y) @ np.abs(f64(wh))) + 2e-5 * (np.abs(y) @ np.abs(f64(wh))) + 1e-6
    assert np.all(np.abs(f64(logits) - ref) <= tol)
