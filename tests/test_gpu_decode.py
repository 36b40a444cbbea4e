"""Decode phase on the GPU: attention of one new query per (batch, head)
against a KV cache, and whole decode steps against the fp64 oracle.  A causal
model's output at position t depends only on tokens 0 .. t, so the oracle runs
the prompt plus the decoded tokens as one sequence and its output at the new
position is the reference for the step."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from tests.gpu_util import DEV, bf16_round, compare, f64, instance_config, sync, to_dev

pytestmark = pytest.mark.gpu

UBF = 2.0 ** -8
U32 = 2.0 ** -24
MAX_ABS, REL_L2 = 2e-2, 1e-2
NAN_BF16 = 0x7FC0


def check(got, ref, what=""):
    ma, rl = compare(got, ref)
    print(f"  {what}: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert np.all(np.isfinite(got))
    assert ma <= MAX_ABS and rl <= REL_L2, (what, ma, rl)


@pytest.mark.parametrize("B,H,n_keys,dh,k_rows,vt_stride", [
    (1, 1, 1, 64, 1, 64),
    (2, 3, 7, 64, 16, 64),
    (3, 2, 513, 64, 600, 640),
    (1, 1, 64, 128, 64, 64),
    (2, 5, 1000, 128, 1000, 1024),
    (1, 3, 1024, 64, 1024, 1024),
    (2, 16, 1025, 128, 1100, 1152),
    (1, 2, 2048, 64, 2048, 2048),           # 32 chunks of 64: the most chunks
    (2, 2, 2049, 64, 2100, 2112),           # first length split into chunks of 256
    (1, 4, 8192, 128, 8192, 8192),
])
def test_decode_attention_kernel(B, H, n_keys, dh, k_rows, vt_stride):
    print(f"decode attention B={B} H={H} keys={n_keys} dh={dh}", flush=True)
    rng = np.random.default_rng(n_keys + dh)
    q = bf16_round(rng.standard_normal((B, H, dh)))
    k = bf16_round(rng.standard_normal((B, H, k_rows, dh)))
    vt = bf16_round(rng.standard_normal((B, H, dh, vt_stride)))
    # cache positions past n_keys hold arbitrary bits: make them NaN
    k.view(torch.int16)[:, :, n_keys:, :] = NAN_BF16
    vt.view(torch.int16)[:, :, :, n_keys:] = NAN_BF16
    ctx = torch.empty((B, H * dh), dtype=torch.bfloat16, device=DEV)
    ie.test_decode_attention(to_dev(q), to_dev(k), to_dev(vt), ctx, B, H, n_keys, dh, k_rows, vt_stride)
    sync()
    q64, k64, v64 = f64(q), f64(k)[:, :, :n_keys], f64(vt)[..., :n_keys]
    # the oracle's attention with the one new query as a length-1 query sequence
    p = F.attention_probs(q64[:, :, None, :], k64, False)[:, :, 0, :]
    ref = F.attention_context(q64[:, :, None, :], k64, np.swapaxes(v64, -1, -2), False).reshape(B, H * dh)
    # fp32 dot products and sums over n_keys terms, then one bf16 rounding
    bound = (dh + 8) * U32 * np.einsum("bhj,bhdj->bhd", p, np.abs(v64)).reshape(B, H * dh) * 4 \
        + (n_keys + 8) * U32 * np.abs(v64).max() + 1e-6
    got = f64(ctx)
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref)
    tol = 1.01 * UBF * np.abs(ref) + bound
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert np.all(err <= tol), (worst, err[worst], tol[worst])


DECODERS = [
    # shape overrides (pre-LN causal), prompt batch, prompt length, decode steps
    (dict(W.STRESS_INIT, n_layers=2, d_model=256, n_heads=4, d_ff=1024, pre_ln=1, causal=1, n_out=2), 3, 37, 4),
    (dict(W.STRESS_INIT, n_layers=2, d_model=256, n_heads=2, d_ff=640, pre_ln=1, causal=1, n_out=0), 2, 64, 3),
    (dict(n_layers=3, d_model=128, n_heads=2, d_ff=512, pre_ln=1, causal=1, n_out=3), 1, 1, 5),
    # batches past 4: the products use fewer K-groups than the packed weight copies were made
    # for, so all four read the row-major weights (6: two K-groups; 12: one, and the fused
    # LayerNorm's waves normalise a second row each)
    (dict(W.STRESS_INIT, n_layers=2, d_model=256, n_heads=4, d_ff=1024, pre_ln=1, causal=1, n_out=2), 6, 20, 3),
    (dict(n_layers=2, d_model=128, n_heads=2, d_ff=512, pre_ln=1, causal=1, n_out=2), 12, 9, 3),
    # decode steps across the 2048 -> 2049 key boundary where the key chunking changes
    (dict(n_layers=1, d_model=128, n_heads=1, d_ff=256, pre_ln=1, causal=1, n_out=2), 2, 2046, 4),
]


@pytest.mark.parametrize("over,B,P,G", DECODERS)
def test_decode_steps_match_oracle(over, B, P, G):
    shape = W.model_shape("encoder_l1_d128_s32_b2", **over)
    d = shape["d_model"]
    print(f"decode {over} B={B} prompt={P} steps={G}", flush=True)
    x = W.make_input(7000 + P, B, P + G, d)
    with ie.Instance(**instance_config(shape, B, P + G + 3), kv_cache=1) as inst:
        inst.submit(torch.from_numpy(x[:, :P].copy()).to(DEV))
        check(inst.read_logits(), F.forward(x[:, :P], shape), "prompt")
        first = None
        for g in range(G):
            xt = torch.from_numpy(np.ascontiguousarray(x[:, P + g])).to(DEV)
            inst.decode(xt, P + g)
            got = inst.read_logits()
            assert got.shape == (B, 1, shape["n_out"] or d)
            check(got[:, 0], F.forward(x[:, :P + g + 1], shape)[:, P + g], f"step {g}")
            if g == 0:
                first = got.copy()
        # rewinding to the first decoded position rewrites the same K and V: same result, bit for bit
        inst.decode(np.ascontiguousarray(x[:, P]), P)      # host input this time
        again = inst.read_logits()
        assert np.array_equal(again.view(np.uint32), first.view(np.uint32))


def test_full_size_decoder_decode():
    name = "decoder_l24_d2048_s1024"
    shape = W.model_shape(name)
    B, P, G = 2, 30, 2
    print(f"decode {name} B={B} prompt={P} steps={G}", flush=True)
    x = W.make_input(W.WORKLOADS[name]["input_seed"], B, P + G, shape["d_model"])
    with ie.Instance(**instance_config(shape, B, 1024), kv_cache=1) as inst:
        inst.submit(torch.from_numpy(x[:, :P].copy()).to(DEV))
        inst.wait()
        for g in range(G):
            inst.decode(torch.from_numpy(np.ascontiguousarray(x[:, P + g])).to(DEV), P + g)
            got = inst.read_logits()
            check(got[:, 0], F.forward(x[:, :P + g + 1], shape)[:, P + g], f"step {g}")


def test_decode_state_errors():
    shape = W.model_shape("encoder_l1_d128_s32_b2", pre_ln=1, causal=1, n_out=2)
    x = W.make_input(1, 2, 8, 128)
    with ie.Instance(**instance_config(shape, 2, 16)) as plain:
        with pytest.raises(ie.IefwdError) as e:
            plain.decode(x[:, 0], 0)                        # no KV cache
        assert e.value.status == ie.ESTATE
    with ie.Instance(**instance_config(shape, 2, 16), kv_cache=1) as inst:
        with pytest.raises(ie.IefwdError) as e:
            inst.decode(x[:, 0], 0)                         # no prompt yet
        assert e.value.status == ie.ESTATE
        inst.submit(x[:, :5].copy())
        inst.wait()
        for bad_pos, bad_x in ((6, x[:, 5]), (16, x[:, 5]), (5, np.zeros((3, 128), np.float32))):
            with pytest.raises(ie.IefwdError) as e:
                inst.decode(np.ascontiguousarray(bad_x), bad_pos)   # past the cache, past max_seq, batch > prompt's
            assert e.value.status == ie.EINVAL
        inst.decode(np.ascontiguousarray(x[:1, 5]), 5)          # fewer sequences than the prompt: fine
        assert inst.read_logits().shape == (1, 1, 2)


SKINNY = [
    # M, N, K, epilogue, LayerNorm activations; K-groups per MFMA in the comments where more than one
    (1, 16, 32, ie.EPI_BIAS_BF16, False),           # one workgroup, one K step
    (16, 768, 96, ie.EPI_BIAS_GELU_BF16, False),    # fewer K steps than waves
    (2, 6144, 2048, ie.EPI_BIAS_BF16, False),       # decoder QKV width: 2 K-groups
    (3, 2048, 8192, ie.EPI_BIAS_RESID_F32, False),  # FFN-down: 4 K-groups
    (7, 128, 4096, ie.EPI_BIAS_GELU_BF16, False),
    (5, 4096, 1056, ie.EPI_BIAS_RESID_F32, False),  # K not a multiple of 64
    (8, 1024, 2048, ie.EPI_BIAS_BF16, False),       # two K-groups, 8 tokens (their limit)
    (4, 2048, 2048, ie.EPI_BIAS_RESID_F32, False),  # four K-groups, 4 tokens (their limit)
    (2, 6144, 2048, ie.EPI_BIAS_BF16, True),
    (16, 1024, 1024, ie.EPI_BIAS_GELU_BF16, True),  # M * K at the prologue's limit
    (4, 512, 4096, ie.EPI_BIAS_RESID_F32, True),    # the longest row; 4 K-groups
    (3, 2304, 768, ie.EPI_BIAS_GELU_BF16, True),    # 2 K-groups (4 would not fit in one round)
    (1, 64, 96, ie.EPI_BIAS_BF16, True),            # a row shorter than 64 lanes x 4
]


@pytest.mark.parametrize("M,N,K,epi,ln", SKINNY)
def test_gemm_skinny(M, N, K, epi, ln):
    """The decode-step product (optionally with its LayerNorm prologue) against
    the oracle's linear layer, LayerNorm and GELU in fp64."""
    print(f"skinny gemm M={M} N={N} K={K} epi={epi} ln={ln}", flush=True)
    rng = np.random.default_rng(M * 1000 + N + K + epi + (7 if ln else 0))
    w = bf16_round(rng.standard_normal((K, N)) * 0.05)                  # [in, out]
    bias = bf16_round(rng.standard_normal(N) * 0.1)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    w64, b64 = f64(w), f64(bias)
    out = torch.empty((M, N), dtype=torch.float32 if epi == ie.EPI_BIAS_RESID_F32 else torch.bfloat16, device=DEV)
    r_d = torch.from_numpy(resid).to(DEV) if epi == ie.EPI_BIAS_RESID_F32 else None
    if ln:
        z = (rng.standard_normal((M, K)) * 2.0 + 0.5).astype(np.float32)
        g = (1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32)
        be = (0.1 * rng.standard_normal(K)).astype(np.float32)
        eps = 1e-5
        ie.test_gemm_skinny(epi, None, to_dev(w.t()), to_dev(bias), r_d, out, M, N, K,
                            ln=(torch.from_numpy(z).to(DEV), torch.from_numpy(g).to(DEV),
                                torch.from_numpy(be).to(DEV), eps))
        z64 = z.astype(np.float64)
        a64 = F.layer_norm(z64, g.astype(np.float64), be.astype(np.float64), eps)
        mean = z64.mean(axis=1, keepdims=True)
        rstd = 1.0 / np.sqrt(z64.var(axis=1, keepdims=True) + eps)
        # fp32 statistics (K-term sums) and the bf16 rounding of the normalised rows
        t = np.abs(g.astype(np.float64)) * rstd * (np.abs(z64 - mean) + np.abs(z64).mean(axis=1, keepdims=True))
        da = 1.01 * UBF * np.abs(a64) + (K + 16) * U32 * t
    else:
        a = bf16_round(rng.standard_normal((M, K)))
        ie.test_gemm_skinny(epi, to_dev(a), to_dev(w.t()), to_dev(bias), r_d, out, M, N, K)
        a64 = f64(a)
        da = np.zeros_like(a64)
    sync()
    pre = F.linear(a64, w64, b64)
    bound = (K + 16) * U32 * ((np.abs(a64) + da) @ np.abs(w64)) + da @ np.abs(w64) + 1e-7
    got = f64(out)
    if epi == ie.EPI_BIAS_BF16:
        ref, tol = pre, bound + 1.01 * UBF * (np.abs(pre) + bound)
    elif epi == ie.EPI_BIAS_GELU_BF16:
        ref = F.gelu(pre)
        tol = 1.13 * bound + 1.01 * UBF * (np.abs(ref) + 1.13 * bound) + 1e-6 * np.abs(pre) + 1e-7
    else:
        ref = pre + resid.astype(np.float64)
        tol = bound + 2 * U32 * (np.abs(ref) + np.abs(resid)) + 1e-7
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got))
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert np.all(err <= tol), f"max excess at {worst}: err {err[worst]} tol {tol[worst]}"


def test_gemm_skinny_rejects():
    w = torch.zeros((64, 64), dtype=torch.bfloat16, device=DEV)
    b = torch.zeros(64, dtype=torch.bfloat16, device=DEV)
    a = torch.zeros((17, 64), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros((17, 64), dtype=torch.bfloat16, device=DEV)
    z = torch.zeros((16, 2048), dtype=torch.float32, device=DEV)
    for args, kw in (((a, w, b, None, out, 17, 64, 64), {}),            # M > 16
                     ((a, w, b, None, out, 2, 40, 64), {}),             # N % 16
                     ((a, w, b, None, out, 2, 64, 48), {}),             # K % 32
                     ((None, w, b, None, out, 16, 64, 2048), {"ln": (z, z[0], z[0], 1e-5)})):  # M * K > 16384
        with pytest.raises(ie.IefwdError) as e:
            ie.test_gemm_skinny(ie.EPI_BIAS_BF16, *args, **kw)
        assert e.value.status == ie.EINVAL
