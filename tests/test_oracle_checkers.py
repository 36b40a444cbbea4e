"""Pins of the oracle functions the GPU parity tests use as their reference or
their acceptance metric: the linear layer, the attention context, and the two
error measures of the acceptance gate (max-abs error and relative L2 error
over a whole output tensor).

Each is checked against something other than itself: a pure-Python triple
loop or the scalar oracle's attention (brute force on tiny inputs), closed
forms (uniform and one-hot attention), and hand-computed numbers.  The shapes
are non-square so that a transposed operand cannot pass.
"""
import math

import numpy as np
import pytest

from oracle import forward as F
from oracle import scalar as SC


def test_linear_matches_triple_loop_on_non_square_shapes():
    rng = np.random.default_rng(11)
    y = rng.standard_normal((3, 5))        # 3 tokens, 5 features in
    w = rng.standard_normal((5, 7))        # logical [in, out]
    b = rng.standard_normal(7)
    got = F.linear(y, w, b)
    ref = np.array(SC.matmul_scalar(y, w)) + b
    assert got.shape == (3, 7)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_linear_bias_is_per_output_column():
    # zero input: every row is the bias itself, in output order
    b = np.array([1.0, -2.0, 3.0, 0.5])
    got = F.linear(np.zeros((2, 3)), np.ones((3, 4)), b)
    np.testing.assert_array_equal(got, np.tile(b, (2, 1)))
    # a one-hot input row selects one row of W (the [in, out] layout)
    w = np.arange(12.0).reshape(3, 4)
    got = F.linear(np.array([[0.0, 1.0, 0.0]]), w, np.zeros(4))
    np.testing.assert_array_equal(got[0], w[1])


def _scalar_context(q, k, v, causal):
    """softmax(q k^T / sqrt(dh)) v written as loops over one head."""
    S, dh = len(q), len(q[0])
    out = []
    for i in range(S):
        n = i + 1 if causal else S
        s = [sum(q[i][t] * k[j][t] for t in range(dh)) / math.sqrt(dh) for j in range(n)]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        tot = sum(e)
        out.append([sum(e[j] / tot * v[j][t] for j in range(n)) for t in range(v.shape[1])])
    return np.array(out)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_context_matches_loops(causal):
    rng = np.random.default_rng(12)
    S, dh = 6, 4
    q, k = rng.standard_normal((S, dh)), rng.standard_normal((S, dh))
    v = rng.standard_normal((S, 3))        # a value width unlike dh and S
    got = F.attention_context(q[None], k[None], v[None], causal)[0]
    np.testing.assert_allclose(got, _scalar_context(q, k, v, causal), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_context_uniform_closed_form(causal):
    # q = 0 makes every score 0: the context of row i is the mean of the
    # value rows it may see (all of them, or rows 0..i when causal)
    rng = np.random.default_rng(13)
    S = 5
    v = rng.standard_normal((S, 4))
    got = F.attention_context(np.zeros((S, 4)), rng.standard_normal((S, 4)), v, causal)
    for i in range(S):
        ref = v[: i + 1].mean(axis=0) if causal else v.mean(axis=0)
        np.testing.assert_allclose(got[i], ref, rtol=1e-14, atol=1e-14)


def test_attention_context_one_hot_selects_value_row():
    # scores of 200 / sqrt(dh) on one key and 0 elsewhere: the weight of the
    # other keys is below e^-90, so row i's context is V[target(i)]
    S, dh = 4, 4
    target = [2, 0, 3, 1]
    q = np.zeros((S, dh))
    k = np.zeros((S, dh))
    for j in range(S):
        k[j, j] = 1.0
    for i, j in enumerate(target):
        q[i, j] = 200.0
    v = np.arange(S * 3, dtype=np.float64).reshape(S, 3) - 4.0
    got = F.attention_context(q, k, v, False)
    np.testing.assert_allclose(got, v[target], rtol=0, atol=1e-30 + 1e-12)


def test_rel_l2_hand_computed():
    ref = np.array([3.0, 4.0])             # |ref| = 5
    got = np.array([3.0, 0.0])             # |got - ref| = 4, |got| = 3
    assert F.rel_l2(got, ref) == pytest.approx(0.8, abs=1e-15)
    # normalised by the reference, not by the result: swapping the arguments
    # divides the same difference by |got| = 3 instead
    assert F.rel_l2(ref, got) == pytest.approx(4.0 / 3.0, abs=1e-15)
    # over the whole tensor, not per row: rows (1, 0) and (0, 2) against (1, 1) and (1, 1)
    got2 = np.array([[1.0, 0.0], [0.0, 2.0]])
    ref2 = np.ones((2, 2))
    assert F.rel_l2(got2, ref2) == pytest.approx(math.sqrt(3.0) / 2.0, abs=1e-15)
    # fp32 inputs are compared in fp64
    assert F.rel_l2(np.float32([1.0 + 2.0 ** -20]), np.array([1.0])) == 2.0 ** -20


def test_max_abs_hand_computed():
    got = np.array([[1.0, -2.0], [0.5, 7.0]])
    ref = np.array([[1.5, -2.0], [-1.0, 6.0]])
    assert F.max_abs(got, ref) == 1.5     # |0.5 - (-1.0)|: the largest, taken with its sign removed
    assert F.max_abs(ref, got) == 1.5
    assert F.max_abs(got, got) == 0.0
    # the largest error sits in the last element of a long vector, with a negative sign
    a = np.zeros(1000)
    b = np.zeros(1000)
    b[-1] = -0.25
    assert F.max_abs(a, b) == 0.25
    # fp32 inputs are compared in fp64
    assert F.max_abs(np.float32([1.0 + 2.0 ** -23]), np.array([1.0])) == 2.0 ** -23
