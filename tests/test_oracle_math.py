"""Pins of the fp64 oracle's arithmetic against brute force, closed forms,
textbook values and invariants (no GPU)."""
import math

import numpy as np
import pytest
from scipy.special import ndtr

import workloads
from oracle import forward as F
from oracle import init_spec as I
from oracle import scalar as SC
from tests.golden_data import rows


# ----------------------------------------------------------------------------- matmul
def test_matmul_vs_triple_loop():
    rng = np.random.default_rng(1)
    a, b = rng.standard_normal((5, 7)), rng.standard_normal((7, 3))
    ref = np.array(SC.matmul_scalar(a, b))
    assert np.max(np.abs(a @ b - ref)) <= 1e-13 * np.abs(a).max() * np.abs(b).max() * 7


# ----------------------------------------------------------------------------- softmax
def test_softmax_rows_sum_to_one_and_shift_invariant():
    rng = np.random.default_rng(2)
    a = rng.standard_normal((6, 9)) * 5
    p = F.softmax_rows(a)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= 1e-12
    assert np.allclose(F.softmax_rows(a + rng.standard_normal((6, 1)) * 10), p, rtol=0, atol=1e-12)
    # two-entry closed form: p0 = 1 / (1 + e^(a1 - a0))
    two = F.softmax_rows(np.array([[0.3, -1.2]]))
    assert two[0, 0] == pytest.approx(1.0 / (1.0 + math.exp(-1.5)), abs=1e-15)


def test_causal_probs_structure():
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
    p = F.attention_probs(q, k, causal=True)
    assert np.all(p[np.triu_indices(5, 1)] == 0.0)           # exactly zero above the diagonal
    assert np.array_equal(p[0], np.eye(5)[0])                  # row 0 attends only to key 0
    assert np.max(np.abs(p.sum(-1) - 1)) <= 1e-12


def test_score_scale_is_inverse_sqrt_dh():
    # dh = 4, q = (1,1,1,1), keys k0 = q, k1 = 0: scores 4/2 = 2 and 0 -> p0 = 1/(1+e^-2)
    q = np.ones((1, 4))
    k = np.array([[1.0, 1, 1, 1], [0, 0, 0, 0]])
    p = F.attention_probs(q, k, causal=False)
    assert p[0, 0] == pytest.approx(1.0 / (1.0 + math.exp(-2.0)), abs=1e-15)


# ----------------------------------------------------------------------------- LayerNorm
def test_layernorm_invariants():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((8, 32)) * 3 + 7
    eps = 1e-5
    y = F.layer_norm(z, np.ones(32), np.zeros(32), eps)
    assert np.max(np.abs(y.mean(-1))) <= 1e-12
    var = z.var(-1)
    assert np.max(np.abs(y.var(-1) - var / (var + eps))) <= 1e-12
    # affine step applied after normalisation
    g, b = rng.standard_normal(32), rng.standard_normal(32)
    assert np.allclose(F.layer_norm(z, g, b, eps), g * y + b, rtol=0, atol=1e-12)
    # constant row -> beta
    c = F.layer_norm(np.full((1, 32), 3.5), g, b, eps)
    assert np.allclose(c, b, rtol=0, atol=1e-15)


# ----------------------------------------------------------------------------- GELU
def test_gelu_textbook_values_and_identities():
    # GELU(u) = u * Phi(u), Phi from the standard normal table (tests/golden/normal_cdf_table.txt)
    for u, phi in ((float(x), float(p)) for x, p in rows("normal_cdf_table.txt")):
        assert F.gelu(np.array(u)) == pytest.approx(u * phi, abs=1e-15)
    u = np.linspace(-6, 6, 241)
    assert np.allclose(F.gelu(u), u * ndtr(u), rtol=0, atol=1e-15)      # library normal CDF
    assert F.gelu(np.array(0.0)) == 0.0
    assert np.allclose(F.gelu(u) - F.gelu(-u), u, rtol=0, atol=1e-14)   # odd part is u/2 * 2
    assert F.gelu(np.array(12.0)) == pytest.approx(12.0, abs=1e-15)


# ----------------------------------------------------------------------------- attention closed forms
def _zero_qk_weights(d, rng):
    w = dict(wqkv=rng.standard_normal((d, 3 * d)), bqkv=rng.standard_normal(3 * d),
             wo=np.eye(d), bo=np.zeros(d))
    w["wqkv"][:, :2 * d] = 0.0
    w["bqkv"][:2 * d] = 0.0
    return w


@pytest.mark.parametrize("causal", [False, True])
def test_uniform_attention_closed_form(causal):
    # Wq = Wk = 0 -> every score 0 -> uniform P: context = mean of the visible V rows
    rng = np.random.default_rng(5)
    B, S, d, H = 2, 6, 8, 2
    y = rng.standard_normal((B, S, d))
    w = _zero_qk_weights(d, rng)
    out = F.self_attention(y, w, H, causal)
    v = y @ w["wqkv"][:, 2 * d:] + w["bqkv"][2 * d:]
    if causal:
        want = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None]
    else:
        want = np.broadcast_to(v.mean(axis=1, keepdims=True), v.shape)
    assert np.allclose(out, want, rtol=0, atol=1e-12)


def test_peaked_attention_selects_one_row():
    # one key dominates by a huge margin -> context = that key's V row
    rng = np.random.default_rng(6)
    S, dh = 5, 4
    q = np.zeros((S, dh)); q[:, 0] = 1.0
    k = np.zeros((S, dh)); k[3, 0] = 2000.0
    v = rng.standard_normal((S, dh))
    p = F.attention_probs(q, k, causal=False)
    assert np.allclose(p @ v, np.broadcast_to(v[3], (S, dh)), rtol=0, atol=1e-12)


def test_heads_use_their_own_columns():
    # head h must read Q/K/V columns [h*dh, (h+1)*dh): permuting heads in the weights
    # permutes the context blocks
    rng = np.random.default_rng(7)
    B, S, d, H = 1, 5, 8, 2
    dh = d // H
    y = rng.standard_normal((B, S, d))
    w = dict(wqkv=rng.standard_normal((d, 3 * d)), bqkv=rng.standard_normal(3 * d),
             wo=np.eye(d), bo=np.zeros(d))
    base = F.self_attention(y, w, H, False)
    perm = np.concatenate([np.arange(dh, 2 * dh), np.arange(0, dh)])
    cols = np.concatenate([perm, d + perm, 2 * d + perm])
    w2 = dict(w, wqkv=w["wqkv"][:, cols], bqkv=w["bqkv"][cols])
    swapped = F.self_attention(y, w2, H, False)
    assert np.allclose(swapped[..., :dh], base[..., dh:], atol=1e-12)
    assert np.allclose(swapped[..., dh:], base[..., :dh], atol=1e-12)


# ----------------------------------------------------------------------------- layer special cases
def _tiny_layer(d, f, rng, zero_branches):
    w = dict(wqkv=rng.standard_normal((d, 3 * d)) * 0.3, bqkv=rng.standard_normal(3 * d) * 0.1,
             wo=rng.standard_normal((d, d)) * 0.3, bo=np.zeros(d),
             ln1_g=1 + 0.1 * rng.standard_normal(d), ln1_b=0.1 * rng.standard_normal(d),
             w1=rng.standard_normal((d, f)) * 0.3, b1=rng.standard_normal(f) * 0.1,
             w2=rng.standard_normal((f, d)) * 0.3, b2=np.zeros(d),
             ln2_g=1 + 0.1 * rng.standard_normal(d), ln2_b=0.1 * rng.standard_normal(d))
    if zero_branches:
        w["wo"][:] = 0.0
        w["w2"][:] = 0.0
    return w


def test_post_ln_with_zero_branches_is_double_ln():
    rng = np.random.default_rng(8)
    d, f = 8, 16
    w = _tiny_layer(d, f, rng, zero_branches=True)
    shape = workloads.tiny_shape(pre_ln=0, causal=0)
    x = rng.standard_normal((2, 4, d))
    out = F.layer(x, w, shape)
    want = F.layer_norm(F.layer_norm(x, w["ln1_g"], w["ln1_b"], 1e-5), w["ln2_g"], w["ln2_b"], 1e-5)
    assert np.allclose(out, want, rtol=0, atol=1e-12)


def test_pre_ln_with_zero_branches_is_identity():
    rng = np.random.default_rng(9)
    d, f = 8, 16
    w = _tiny_layer(d, f, rng, zero_branches=True)
    shape = workloads.tiny_shape(pre_ln=1, causal=1)
    x = rng.standard_normal((2, 4, d))
    assert np.array_equal(F.layer(x, w, shape), x)


def test_post_ln_output_rows_are_normalised():
    # with gamma = 1, beta = 0 every post-LN output row has mean 0 and var ~ 1
    rng = np.random.default_rng(10)
    d, f = 16, 32
    w = _tiny_layer(d, f, rng, zero_branches=False)
    w.update(ln2_g=np.ones(d), ln2_b=np.zeros(d))
    shape = workloads.tiny_shape(pre_ln=0, causal=0, d_model=d, d_ff=f)
    out = F.layer(rng.standard_normal((2, 5, d)), w, shape)
    assert np.max(np.abs(out.mean(-1))) <= 1e-12
    assert np.max(np.abs(out.var(-1) - 1.0)) <= 1e-3


# ----------------------------------------------------------------------------- whole model
@pytest.mark.parametrize("pre_ln,causal,n_out", [(0, 0, 0), (0, 0, 2), (1, 1, 2), (1, 0, 0), (0, 1, 2)])
def test_numpy_oracle_matches_scalar_oracle(oracle_built, pre_ln, causal, n_out):
    shape = workloads.tiny_shape(pre_ln=pre_ln, causal=causal, n_out=n_out)
    x = workloads.make_input(17, 2, 4, shape["d_model"])
    got = F.forward(x, shape)
    want = np.array(SC.forward_scalar(x, shape, lambda l: I.ref_layer_weights(shape, l),
                                      I.global_weights(shape)))
    assert got.shape == want.shape
    assert np.max(np.abs(got - want)) <= 1e-12 * max(1.0, np.abs(want).max())


def test_causal_prefix_property(oracle_built):
    # causal stack: outputs at positions < p do not depend on tokens >= p
    shape = workloads.tiny_shape(pre_ln=1, causal=1, n_out=2)
    x = workloads.make_input(18, 2, 6, shape["d_model"])
    y = x.copy()
    y[:, 4:] = workloads.make_input(19, 2, 2, shape["d_model"])
    a, b = F.forward(x, shape), F.forward(y, shape)
    assert np.array_equal(a[:, :4], b[:, :4])
    assert not np.allclose(a[:, 4:], b[:, 4:])


def test_bidirectional_permutation_equivariance(oracle_built):
    # no positions and no mask: permuting a sequence's tokens permutes its outputs
    shape = workloads.tiny_shape(pre_ln=0, causal=0, n_out=2)
    x = workloads.make_input(20, 2, 5, shape["d_model"])
    perm = np.array([3, 0, 4, 1, 2])
    a, b = F.forward(x, shape), F.forward(x[:, perm], shape)
    assert np.allclose(b, a[:, perm], rtol=0, atol=1e-12)


def test_sequences_are_independent(oracle_built):
    shape = workloads.tiny_shape(pre_ln=0, causal=0, n_out=2)
    x = workloads.make_input(21, 3, 4, shape["d_model"])
    full = F.forward(x, shape)
    one = F.forward(x[1:2], shape)
    assert np.array_equal(full[1:2], one)


def test_head_is_per_token_linear(oracle_built):
    shape = workloads.tiny_shape(pre_ln=0, causal=0, n_out=2)
    x = workloads.make_input(22, 1, 4, shape["d_model"])
    hid = F.forward(x, dict(shape, n_out=0))
    g = I.global_weights(shape)
    want = np.array(SC.matmul_scalar(hid[0], g["wh"])) + g["bh"]
    assert np.allclose(F.forward(x, shape)[0], want, rtol=0, atol=1e-12)
