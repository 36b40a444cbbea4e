"""Pure-Python scalar forward pass for tiny shapes (test infrastructure only).

An independent second implementation of the same definitions as
``oracle.forward`` -- nested loops over Python floats, no NumPy arithmetic --
used to pin the NumPy oracle on shapes like B=2, S=4, d=8.  Same readings of
the points the paper leaves open (see ``oracle.forward``).
"""
from __future__ import annotations

import math


def _matvec_rows(x, w, b):
    """rows of x [n][k] times w [k][m] plus b [m]"""
    k_dim, m_dim = len(w), len(w[0])
    out = []
    for row in x:
        o = []
        for j in range(m_dim):
            acc = 0.0
            for k in range(k_dim):
                acc += row[k] * w[k][j]
            o.append(acc + b[j])
        out.append(o)
    return out


def _ln_row(z, g, b, eps):
    n = len(z)
    mu = sum(z) / n
    var = sum((v - mu) * (v - mu) for v in z) / n
    inv = 1.0 / math.sqrt(var + eps)
    return [g[i] * (z[i] - mu) * inv + b[i] for i in range(n)]


def _gelu(u):
    return 0.5 * u * (1.0 + math.erf(u / math.sqrt(2.0)))


def _attention_seq(y, w, n_heads, causal):
    """one sequence y [S][d] -> Attn(y) [S][d]"""
    S, d = len(y), len(y[0])
    dh = d // n_heads
    qkv = _matvec_rows(y, w["wqkv"], w["bqkv"])
    ctx = [[0.0] * d for _ in range(S)]
    for h in range(n_heads):
        qo, ko, vo = h * dh, d + h * dh, 2 * d + h * dh
        for i in range(S):
            n_keys = i + 1 if causal else S
            scores = []
            for j in range(n_keys):
                dot = 0.0
                for t in range(dh):
                    dot += qkv[i][qo + t] * qkv[j][ko + t]
                scores.append(dot / math.sqrt(dh))
            m = max(scores)
            ex = [math.exp(s - m) for s in scores]
            tot = sum(ex)
            for t in range(dh):
                acc = 0.0
                for j in range(n_keys):
                    acc += ex[j] / tot * qkv[j][vo + t]
                ctx[i][h * dh + t] = acc
    return _matvec_rows(ctx, w["wo"], w["bo"])


def _ffn_seq(y, w):
    hid = _matvec_rows(y, w["w1"], w["b1"])
    hid = [[_gelu(v) for v in row] for row in hid]
    return _matvec_rows(hid, w["w2"], w["b2"])


def _add(a, b):
    return [[a[i][j] + b[i][j] for j in range(len(a[0]))] for i in range(len(a))]


def _ln_rows(x, g, b, eps):
    return [_ln_row(r, g, b, eps) for r in x]


def _tolist(a):
    return a.tolist() if hasattr(a, "tolist") else a


def forward_scalar(x, shape, layer_w, global_w):
    """x: nested lists or an array [B][S][d]; weights as dicts of arrays/lists.
    Returns nested lists [B][S][n_out or d]."""
    x = _tolist(x)
    eps, H, causal = shape["ln_eps"], shape["n_heads"], bool(shape["causal"])
    out = []
    for seq in x:
        h = [list(map(float, r)) for r in seq]
        for l in range(shape["n_layers"]):
            w = {k: _tolist(v) for k, v in layer_w(l).items()}
            if shape["pre_ln"]:
                h1 = _add(h, _attention_seq(_ln_rows(h, w["ln1_g"], w["ln1_b"], eps), w, H, causal))
                h = _add(h1, _ffn_seq(_ln_rows(h1, w["ln2_g"], w["ln2_b"], eps), w))
            else:
                h1 = _ln_rows(_add(h, _attention_seq(h, w, H, causal)), w["ln1_g"], w["ln1_b"], eps)
                h = _ln_rows(_add(h1, _ffn_seq(h1, w)), w["ln2_g"], w["ln2_b"], eps)
        g = {k: _tolist(v) for k, v in global_w.items()}
        if shape["pre_ln"]:
            h = _ln_rows(h, g["lnf_g"], g["lnf_b"], eps)
        if shape["n_out"] > 0:
            h = _matvec_rows(h, g["wh"], g["bh"])
        out.append(h)
    return out


def matmul_scalar(a, b):
    """triple loop a [n][k] @ b [k][m]"""
    a, b = _tolist(a), _tolist(b)
    n, k_dim, m = len(a), len(b), len(b[0])
    return [[sum(a[i][k] * b[k][j] for k in range(k_dim)) for j in range(m)] for i in range(n)]
