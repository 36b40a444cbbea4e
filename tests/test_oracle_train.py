"""Pins of the training-step oracle (oracle/train.py) against what the
mathematics fixes: central finite differences of the fp64 forward for every
gradient element of a tiny model, closed forms of the cross-entropy, and
PyTorch's own AdamW (a library routine) for the optimiser."""
import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import train as T

TINY = dict(n_layers=2, d_model=8, n_heads=2, d_ff=16, pre_ln=0, causal=0, n_out=3, ln_eps=1e-5,
            w_std=0.3, b_std=0.1, ln_std=0.1, qk_std=0.5, seed=11)


def tiny_params(shape):
    return T.initial_params(shape)


def flat(tree):
    out = []
    for l, w in enumerate(tree["layers"]):
        for k in T.LAYER_PARAMS:
            out.append((("layers", l, k), w[k]))
    for k in T.HEAD_PARAMS:
        out.append(((k,), tree[k]))
    return out


def get(tree, path):
    return tree["layers"][path[1]][path[2]] if path[0] == "layers" else tree[path[0]]


@pytest.mark.parametrize("causal", [0, 1])
def test_gradients_match_finite_differences(causal):
    shape = dict(TINY, causal=causal, n_layers=2 if not causal else 1)
    params = tiny_params(shape)
    x = W.make_input(5, 2, 4, shape["d_model"]).astype(np.float64)
    labels = W.make_labels(6, 2, 4, shape["n_out"])
    loss, grads, dx = T.loss_and_grads(params, x, labels, shape)
    assert abs(loss - T.loss_only(params, x, labels, shape)) < 1e-12
    h = 1e-6
    worst = 0.0
    for path, w in flat(params):
        g = get(grads, path)
        assert g.shape == w.shape, path
        it = np.nditer(w, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            old = w[i]
            w[i] = old + h
            lp = T.loss_only(params, x, labels, shape)
            w[i] = old - h
            lm = T.loss_only(params, x, labels, shape)
            w[i] = old
            fd = (lp - lm) / (2 * h)
            err = abs(fd - g[i])
            worst = max(worst, err)
            assert err <= 1e-7 + 1e-6 * abs(fd), (path, i, fd, g[i])
    # the input gradient too (the first layer's dX)
    for i in [(0, 0, 0), (1, 3, 7), (0, 2, 5)]:
        xp, xm = x.copy(), x.copy()
        xp[i] += h
        xm[i] -= h
        fd = (T.loss_only(params, xp, labels, shape) - T.loss_only(params, xm, labels, shape)) / (2 * h)
        assert abs(fd - dx[i]) <= 1e-7 + 1e-6 * abs(fd)


def test_cross_entropy_closed_forms():
    labels = np.array([[0, 2, 1]])
    loss, d = T.cross_entropy(np.zeros((1, 3, 4)), labels)
    assert abs(loss - math.log(4)) < 1e-15                  # uniform logits: ln(classes)
    assert np.allclose(d.sum(axis=-1), 0.0, atol=1e-16)     # softmax - onehot sums to 0 per row
    assert np.allclose(d[0, 0], np.array([-0.75, 0.25, 0.25, 0.25]) / 3)
    big = np.zeros((1, 1, 2))
    big[0, 0, 1] = 50.0
    loss, _ = T.cross_entropy(big, np.array([[1]]))
    assert 0 <= loss < 1e-20                                # confident and right: ~ e^-50 (below fp64 resolution)
    loss, _ = T.cross_entropy(big, np.array([[0]]))
    assert abs(loss - 50.0) < 1e-12                         # confident and wrong: the margin


@pytest.mark.parametrize("decay", [True, False])
def test_adamw_matches_torch(decay):
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal((5, 7))
    hp = dict(lr=3e-3, beta1=0.85, beta2=0.99, eps=1e-7, weight_decay=0.05)
    w, m, v = w0.copy(), np.zeros_like(w0), np.zeros_like(w0)
    tw = torch.tensor(w0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([tw], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
                            weight_decay=hp["weight_decay"] if decay else 0.0)
    for step in range(1, 8):
        g = rng.standard_normal(w0.shape) * (0.1 if step % 2 else 3.0)
        w, m, v = T.adamw_update(w, g, m, v, step, decay, **hp)
        tw.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        assert np.allclose(w, tw.detach().numpy(), rtol=0, atol=1e-14), step


def test_training_reduces_the_loss():
    shape = dict(TINY, n_layers=1)
    params = tiny_params(shape)
    opt = T.AdamW(params, lr=3e-2, weight_decay=0.0)
    x = W.make_input(8, 2, 4, shape["d_model"]).astype(np.float64)
    labels = W.make_labels(9, 2, 4, shape["n_out"])
    losses = [T.train_step(params, opt, x, labels, shape) for _ in range(30)]
    assert losses[-1] < 0.5 * losses[0]
    assert opt.step_no == 30


def test_post_ln_only():
    shape = dict(TINY, pre_ln=1)
    with pytest.raises(ValueError):
        T.loss_and_grads(tiny_params(shape), np.zeros((1, 2, 8)), np.zeros((1, 2), np.int32), shape)
