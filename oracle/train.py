"""Oracle for one training step of a post-LN encoder (the BERT-base-shaped
model of a training function co-located with inference, Sec. 5.1 and 5.2),
written out plainly in fp64.

Test infrastructure only (see oracle/__init__.py): nothing in the product
imports it.

The paper trains its models with a DL framework and states none of the
arithmetic of a training step.  This file writes out the standard
definitions, with the readings of what the paper leaves open (each also
listed in the design notes):

  T1  model: the post-LN encoder of ``forward.layer`` (bidirectional or causal
      attention), per-token head X_L W_h + b_h with n_out classes.
  T2  loss: mean over all B*S tokens of the softmax cross-entropy of the
      token's logits against an integer label in [0, n_out).
  T3  optimiser: AdamW (decoupled weight decay, bias-corrected moments):
        m <- b1 m + (1 - b1) g;   v <- b2 v + (1 - b2) g^2
        w <- w (1 - lr wd) - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
      weight decay only on the weight matrices (not on biases or LayerNorm
      gamma / beta); defaults lr 1e-4, b1 0.9, b2 0.999, eps 1e-8, wd 0.01.
  T4  one step = forward, loss, backward of every parameter, one AdamW update;
      no gradient clipping, no dropout, no learning-rate schedule.

Backward, per post-LN layer (X input, forward z1 = X + Attn(X), X1 = LN1(z1),
v = X1 W1 + b1, u = GELU(v), z2 = X1 + u W2 + b2, X' = LN2(z2)):
  LN backward:  x^ = (z - mean) * rstd,  g = dY * gamma,
                dz = rstd * (g - mean(g) - x^ * mean(g * x^)),
                dgamma = sum_rows dY * x^,  dbeta = sum_rows dY
  linear y = a W + b:  da = dy W^T,  dW = a^T dy,  db = sum_rows dy
  GELU:  du/dv = Phi(v) + v phi(v)
  attention (per head, S = q k^T / sqrt(dh), P = softmax(S), C = P v):
                dv = P^T dC,  dP = dC v^T,  dS = P * (dP - rowsum(dP * P)),
                dq = dS k / sqrt(dh),  dk = dS^T q / sqrt(dh)
  softmax cross-entropy (per token, N tokens):  dlogits = (softmax - onehot) / N
These are pinned against central finite differences of the fp64 forward on a
tiny model (tests/test_oracle_train.py), which checks every gradient element.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from . import forward as F
from . import init_spec

ADAMW_DEFAULTS = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
# parameters that take weight decay (the weight matrices)
DECAYED = ("wqkv", "wo", "w1", "w2", "wh")
LAYER_PARAMS = ("wqkv", "bqkv", "wo", "bo", "ln1_g", "ln1_b", "w1", "b1", "w2", "b2", "ln2_g", "ln2_b")
HEAD_PARAMS = ("wh", "bh")


def initial_params(shape: dict) -> dict:
    """fp64 copies of the seeded init: {"layers": [dict per layer], "wh", "bh"}."""
    g = init_spec.global_weights(shape)
    return {"layers": [init_spec.layer_weights(shape, l) for l in range(shape["n_layers"])],
            "wh": g["wh"], "bh": g["bh"]}


# ------------------------------------------------------------------ pieces with caches
def _ln_fwd(z, gamma, beta, eps):
    mean = z.mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(((z - mean) ** 2).mean(axis=-1, keepdims=True) + eps)
    xhat = (z - mean) * rstd
    return gamma * xhat + beta, (xhat, rstd)


def _ln_bwd(dy, gamma, cache):
    xhat, rstd = cache
    g = dy * gamma
    dz = rstd * (g - g.mean(axis=-1, keepdims=True) - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    axes = tuple(range(dy.ndim - 1))
    return dz, (dy * xhat).sum(axis=axes), dy.sum(axis=axes)


def _gelu_grad(v):
    phi = np.exp(-0.5 * v * v) / math.sqrt(2.0 * math.pi)
    return 0.5 * (1.0 + erf(v / math.sqrt(2.0))) + v * phi


def _heads(t, n_heads):
    B, S, d = t.shape
    return t.reshape(B, S, n_heads, d // n_heads).transpose(0, 2, 1, 3)


def _merge(t):
    B, H, S, dh = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B, S, H * dh)


def _attn_fwd(y, w, n_heads, causal):
    d = y.shape[-1]
    qkv = y @ w["wqkv"] + w["bqkv"]
    q, k, v = (_heads(qkv[..., i * d:(i + 1) * d], n_heads) for i in range(3))
    p = F.attention_probs(q, k, causal)
    ctx = _merge(p @ v)
    return ctx @ w["wo"] + w["bo"], (y, q, k, v, p, ctx)


def _attn_bwd(dout, w, n_heads, cache):
    """Gradients of Attn(Y) for dout = dL/dAttn(Y)."""
    y, q, k, v, p, ctx = cache
    grads = {}
    axes = tuple(range(dout.ndim - 1))
    grads["wo"] = ctx.reshape(-1, ctx.shape[-1]).T @ dout.reshape(-1, dout.shape[-1])
    grads["bo"] = dout.sum(axis=axes)
    dctx = _heads(dout @ w["wo"].T, n_heads)                 # [B, H, S, dh]
    dh = q.shape[-1]
    dv = np.swapaxes(p, -1, -2) @ dctx
    dp = dctx @ np.swapaxes(v, -1, -2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = (ds @ k) / math.sqrt(dh)
    dk = (np.swapaxes(ds, -1, -2) @ q) / math.sqrt(dh)
    dqkv = np.concatenate([_merge(dq), _merge(dk), _merge(dv)], axis=-1)     # [B, S, 3d]
    grads["wqkv"] = y.reshape(-1, y.shape[-1]).T @ dqkv.reshape(-1, dqkv.shape[-1])
    grads["bqkv"] = dqkv.sum(axis=axes)
    return dqkv @ w["wqkv"].T, grads


def layer_forward(x, w, shape):
    """Post-LN layer with everything its backward needs."""
    eps, H, causal = shape["ln_eps"], shape["n_heads"], bool(shape["causal"])
    att, c_att = _attn_fwd(x, w, H, causal)
    x1, c_ln1 = _ln_fwd(x + att, w["ln1_g"], w["ln1_b"], eps)
    vpre = x1 @ w["w1"] + w["b1"]
    u = F.gelu(vpre)
    x2, c_ln2 = _ln_fwd(x1 + u @ w["w2"] + w["b2"], w["ln2_g"], w["ln2_b"], eps)
    return x2, (c_att, x1, c_ln1, vpre, u, c_ln2)


def layer_backward(dx2, w, shape, cache):
    """dL/dX and the layer's parameter gradients, for dx2 = dL/dX'."""
    c_att, x1, c_ln1, vpre, u, c_ln2 = cache
    g = {}
    dz2, g["ln2_g"], g["ln2_b"] = _ln_bwd(dx2, w["ln2_g"], c_ln2)
    rows = lambda t: t.reshape(-1, t.shape[-1])
    g["w2"] = rows(u).T @ rows(dz2)
    g["b2"] = rows(dz2).sum(axis=0)
    dvpre = (dz2 @ w["w2"].T) * _gelu_grad(vpre)
    g["w1"] = rows(x1).T @ rows(dvpre)
    g["b1"] = rows(dvpre).sum(axis=0)
    dx1 = dz2 + dvpre @ w["w1"].T
    dz1, g["ln1_g"], g["ln1_b"] = _ln_bwd(dx1, w["ln1_g"], c_ln1)
    dy, ga = _attn_bwd(dz1, w, shape["n_heads"], c_att)
    g.update(ga)
    return dz1 + dy, g


def cross_entropy(logits, labels):
    """Mean softmax cross-entropy over tokens and dL/dlogits."""
    n_tok = labels.size
    m = logits.max(axis=-1, keepdims=True)
    lse = m + np.log(np.exp(logits - m).sum(axis=-1, keepdims=True))
    onehot = np.eye(logits.shape[-1])[labels]
    loss = float((lse - (logits * onehot).sum(axis=-1, keepdims=True)).sum() / n_tok)
    return loss, (np.exp(logits - lse) - onehot) / n_tok


def loss_and_grads(params, x, labels, shape):
    """Forward, loss and every parameter's gradient for fp32 inputs x [B, S, d]
    and integer labels [B, S]."""
    if shape["pre_ln"]:
        raise ValueError("the training oracle covers post-LN stacks")
    h = np.asarray(x, dtype=np.float64)
    caches = []
    for w in params["layers"]:
        h, c = layer_forward(h, w, shape)
        caches.append(c)
    logits = h @ params["wh"] + params["bh"]
    loss, dlogits = cross_entropy(logits, np.asarray(labels))
    rows = lambda t: t.reshape(-1, t.shape[-1])
    grads = {"wh": rows(h).T @ rows(dlogits), "bh": rows(dlogits).sum(axis=0), "layers": [None] * len(caches)}
    dh = dlogits @ params["wh"].T
    for l in reversed(range(len(caches))):
        dh, grads["layers"][l] = layer_backward(dh, params["layers"][l], shape, caches[l])
    return loss, grads, dh


def loss_only(params, x, labels, shape) -> float:
    h = np.asarray(x, dtype=np.float64)
    for w in params["layers"]:
        h = F.layer(h, w, shape)
    return cross_entropy(h @ params["wh"] + params["bh"], np.asarray(labels))[0]


# ------------------------------------------------------------------ AdamW
def adamw_update(w, g, m, v, step, decay, lr, beta1, beta2, eps, weight_decay):
    """One AdamW update (step t = step >= 1); returns new (w, m, v)."""
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    w = w * (1.0 - lr * weight_decay) if decay else w
    return w - lr * mhat / (np.sqrt(vhat) + eps), m, v


class AdamW:
    """Optimiser state over the parameter tree of ``initial_params``."""

    def __init__(self, params, **hp):
        self.hp = dict(ADAMW_DEFAULTS, **hp)
        self.step_no = 0
        zeros = lambda t: {k: np.zeros_like(v) for k, v in t.items()}
        self.m = {"layers": [zeros(w) for w in params["layers"]], "wh": np.zeros_like(params["wh"]),
                  "bh": np.zeros_like(params["bh"])}
        self.v = {"layers": [zeros(w) for w in params["layers"]], "wh": np.zeros_like(params["wh"]),
                  "bh": np.zeros_like(params["bh"])}

    def apply(self, params, grads):
        self.step_no += 1
        hp = self.hp
        for l, w in enumerate(params["layers"]):
            for k in LAYER_PARAMS:
                w[k], self.m["layers"][l][k], self.v["layers"][l][k] = adamw_update(
                    w[k], grads["layers"][l][k], self.m["layers"][l][k], self.v["layers"][l][k], self.step_no,
                    k in DECAYED, **hp)
        for k in HEAD_PARAMS:
            params[k], self.m[k], self.v[k] = adamw_update(params[k], grads[k], self.m[k], self.v[k], self.step_no,
                                                           k in DECAYED, **hp)


def train_step(params, opt: AdamW, x, labels, shape) -> float:
    """One training step in place; returns the step's loss (before the update)."""
    loss, grads, _ = loss_and_grads(params, x, labels, shape)
    opt.apply(params, grads)
    return loss
