"""Plain NumPy fp64 forward pass of one serverless DL instance (the oracle proper).

Test infrastructure only (see the package docstring).

The paper's instances run BERT-base / RoBERTa-large / GPT2-large class models
through a DL framework (Sec. 5.1 "Workloads"); it gives none of the
arithmetic.  This file writes out the standard transformer definitions, with the
readings of the points the paper leaves open:

* LN(z) = gamma * (z - mean) / sqrt(var + eps) + beta, biased variance, eps 1e-5.
* GELU(u) = u/2 * (1 + erf(u / sqrt 2))  (exact erf form).
* attention: scores Q K^T / sqrt(dh); causal keeps keys j <= i; no padding mask;
  no dropout (inference).
* post-LN layer:  X1 = LN1(X + Attn(X));      X' = LN2(X1 + FFN(X1)).
* pre-LN layer:   X1 = X + Attn(LN1(X));      X' = X1 + FFN(LN2(X1));
  a final LN_f after the last layer of a pre-LN stack.
* output: per-token linear head X_L W_h + b_h when n_out > 0, else X_L.
* inputs are the fp32 embeddings themselves: no embedding LN, no positions.

Every weight is the exact fp64 value of the stored bf16 (or fp32 LN) number.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

from . import init_spec


def layer_norm(z: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return gamma * ((z - mu) / np.sqrt(var + eps)) + beta


def gelu(u: np.ndarray) -> np.ndarray:
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def softmax_rows(a: np.ndarray) -> np.ndarray:
    """Softmax over the last axis; -inf entries get probability exactly 0."""
    m = a.max(axis=-1, keepdims=True)
    e = np.exp(a - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention_probs(q: np.ndarray, k: np.ndarray, causal: bool) -> np.ndarray:
    """P = softmax(q k^T / sqrt(dh) [+ causal mask]) for q, k of shape [..., S, dh]."""
    dh = q.shape[-1]
    a = (q @ np.swapaxes(k, -1, -2)) / math.sqrt(dh)
    if causal:
        s = a.shape[-1]
        above = np.triu(np.ones((s, s), dtype=bool), k=1)     # j > i
        a = np.where(above, -np.inf, a)
    return softmax_rows(a)


def linear(y: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y W + b with W in the logical [in, out] layout."""
    return y @ w + b


def attention_context(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal: bool) -> np.ndarray:
    """softmax(q k^T / sqrt(dh) [+ causal]) v for [..., S, dh] operands."""
    return attention_probs(q, k, causal) @ v


def self_attention(y: np.ndarray, w: dict, n_heads: int, causal: bool) -> np.ndarray:
    """Attn(Y) for Y of shape [B, S, d]: fused QKV projection, per-head
    softmax attention, heads concatenated, output projection."""
    B, S, d = y.shape
    dh = d // n_heads
    qkv = y @ w["wqkv"] + w["bqkv"]                     # [B, S, 3d]; columns Q | K | V
    q, k, v = qkv[..., :d], qkv[..., d:2 * d], qkv[..., 2 * d:]

    def heads(t):                                        # [B, S, d] -> [B, H, S, dh]
        return t.reshape(B, S, n_heads, dh).transpose(0, 2, 1, 3)

    p = attention_probs(heads(q), heads(k), causal)       # [B, H, S, S]
    c = p @ heads(v)                                      # [B, H, S, dh]
    c = c.transpose(0, 2, 1, 3).reshape(B, S, d)          # concat heads
    return c @ w["wo"] + w["bo"]


def ffn(y: np.ndarray, w: dict) -> np.ndarray:
    return gelu(y @ w["w1"] + w["b1"]) @ w["w2"] + w["b2"]


def layer(x: np.ndarray, w: dict, shape: dict) -> np.ndarray:
    eps, H, causal = shape["ln_eps"], shape["n_heads"], bool(shape["causal"])
    if shape["pre_ln"]:
        x1 = x + self_attention(layer_norm(x, w["ln1_g"], w["ln1_b"], eps), w, H, causal)
        return x1 + ffn(layer_norm(x1, w["ln2_g"], w["ln2_b"], eps), w)
    x1 = layer_norm(x + self_attention(x, w, H, causal), w["ln1_g"], w["ln1_b"], eps)
    return layer_norm(x1 + ffn(x1, w), w["ln2_g"], w["ln2_b"], eps)


def finish(x: np.ndarray, g: dict, shape: dict) -> np.ndarray:
    """Final LN (pre-LN stacks only) and the optional per-token head."""
    if shape["pre_ln"]:
        x = layer_norm(x, g["lnf_g"], g["lnf_b"], shape["ln_eps"])
    if shape["n_out"] > 0:
        return x @ g["wh"] + g["bh"]
    return x


def forward_with(x: np.ndarray, shape: dict, layer_w, global_w: dict) -> np.ndarray:
    """Forward with explicit weights: ``layer_w(l)`` returns layer l's dict."""
    h = np.asarray(x, dtype=np.float64)
    for l in range(shape["n_layers"]):
        h = layer(h, layer_w(l), shape)
    return finish(h, global_w, shape)


def forward(x: np.ndarray, shape: dict) -> np.ndarray:
    """fp64 output [B, S, n_out] (or [B, S, d] when n_out == 0) for fp32 input x.

    Weights come from the seeded init spec, generated one layer at a time so
    that large stacks do not hold every fp64 layer at once."""
    return forward_with(x, shape, lambda l: init_spec.layer_weights(shape, l),
                        init_spec.global_weights(shape))


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(np.asarray(got, np.float64) - ref) / np.linalg.norm(ref))


def max_abs(got: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64))))
