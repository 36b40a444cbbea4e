"""Pins of the oracle's random-init spec against things other than itself:
published generator outputs, a library bf16 cast, exact arithmetic and the
normal distribution's moments."""
import math

import numpy as np
import pytest
import torch

from oracle import init_spec as I


def test_splitmix64_published_vectors(oracle_built):
    # SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) started from state 0 emits
    # 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F -- the outputs
    # of the published reference implementation.  mix64(z) is the output
    # function taken from state z, so outputs k = mix64(k * golden).
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    for k, w in enumerate(want):
        z = (k * I.GOLDEN) & I.MASK64
        assert I.ref_mix64(z) == w
        assert I.mix64(z) == w


def test_key_derivation_matches_reference(oracle_built):
    for seed in (0, 1, 2, 2**63 + 5, 2**64 - 1):
        for layer in (0, 3, 24):
            for slot in range(16):
                assert I.tensor_key(seed, layer, slot) == I.ref_tensor_key(seed, layer, slot)


def test_box_muller_special_values():
    # u1 = 1 (a>>11 = 2^53 - 1) gives n = 0 for every u2; u2 = 0 gives n = sqrt(-2 ln u1).
    # Check through the definition's two branches with hand-built uniforms.
    assert math.sqrt(-2.0 * math.log(1.0)) * math.cos(0.3) == 0.0
    u1 = 0.25
    assert math.sqrt(-2.0 * math.log(u1)) * math.cos(0.0) == pytest.approx(math.sqrt(4 * math.log(2)), abs=1e-15)


def test_normals_moments(oracle_built):
    # 2e6 draws of a standard normal: mean 0, variance 1, kurtosis 3, P(|n|<1)=0.6827
    n = I.std_normals(I.tensor_key(123, 0, 0), 2_000_000)
    se = 1.0 / math.sqrt(n.size)
    assert abs(n.mean()) < 5 * se
    assert abs(n.var() - 1.0) < 5 * math.sqrt(2) * se
    assert abs((n ** 4).mean() - 3.0) < 5 * math.sqrt(96) * se
    assert abs((np.abs(n) < 1).mean() - 0.682689492) < 5 * 0.47 * se


def test_fast_normals_equal_reference(oracle_built):
    key = I.tensor_key(99, 1, 6)
    fast = I.std_normals(key, 500)
    ref = np.array([I.ref_std_normal(key, e) for e in range(500)])
    assert np.array_equal(fast, ref)


@pytest.mark.parametrize("seed", [1, 2, 12345])
def test_bf16_fast_path_equals_reference(oracle_built, seed):
    # C fast path (bit trick) vs pure-Python path (exact rational rounding)
    fast = I.gen_weight(seed, 2, I.SLOTS["wqkv"], 8, 24, 0.02, qk_cols=16, sigma_qk=0.06)
    ref = I.ref_weight(seed, 2, I.SLOTS["wqkv"], 8, 24, 0.02, qk_cols=16, sigma_qk=0.06)
    assert np.array_equal(fast, ref)
    g_fast = I.gen_ln_param(seed, 0, I.SLOTS["ln1_g"], 40, 1.0, 0.02)
    g_ref = I.ref_ln_param(seed, 0, I.SLOTS["ln1_g"], 40, 1.0, 0.02)
    assert np.array_equal(g_fast, g_ref)


def test_bf16_rounding_against_library_cast():
    # RNE fp32 -> bf16 of the exact-arithmetic reference equals torch's CPU cast
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 0.05,
        # exact ties: bf16 value plus half a quantum, both parities of the kept LSB
        (np.array([1.0, 1.0078125, 2.0, -3.0], np.float32)
         + np.array([2.0 ** -8, 2.0 ** -8, 2.0 ** -7, -(2.0 ** -7)], np.float32)),
    ]).astype(np.float32)
    lib = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    ref = np.array([I.ref_round_bf16(float(v)) for v in vals])
    assert np.array_equal(lib, ref)
    # hand-checked ties: 1 + 2^-8 sits halfway between 1 and 1 + 2^-7 -> even (1.0)
    assert I.ref_round_bf16(1.0 + 2.0 ** -8) == 1.0
    # 1 + 3*2^-8 is halfway between 1+2^-7 (odd) and 1+2^-6 (even) -> 1+2^-6
    assert I.ref_round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6


def test_fast_bits_match_library_rounding(oracle_built):
    # the bf16 produced by the C path equals torch's RNE cast of the fp32 value
    key = I.tensor_key(5, 0, I.SLOTS["w1"])
    n = I.std_normals(key, 4096)
    f32 = (0.02 * n).astype(np.float32)
    want = torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = I.gen_weight_bits(5, 0, I.SLOTS["w1"], 64, 64, 0.02).reshape(-1)
    assert np.array_equal(got, want)


def test_default_init_is_exact_identity_affine(oracle_built):
    # b_std = ln_std = 0: biases are zeros (+-0), gamma = 1, beta = 0 exactly
    b = I.gen_weight(3, 0, I.SLOTS["b1"], 1, 64, 0.0)
    assert np.all(b == 0.0)
    g = I.gen_ln_param(3, 0, I.SLOTS["ln1_g"], 64, 1.0, 0.0)
    assert np.all(g == 1.0)
    be = I.gen_ln_param(3, 0, I.SLOTS["ln1_b"], 64, 0.0, 0.0)
    assert np.all(be == 0.0)


def test_qk_block_uses_its_own_sigma(oracle_built):
    w = I.gen_weight(11, 0, I.SLOTS["wqkv"], 256, 96, 0.02, qk_cols=64, sigma_qk=0.2)
    assert 0.17 < w[:, :64].std() < 0.23
    assert 0.017 < w[:, 64:].std() < 0.023


def test_weight_std_and_independence(oracle_built):
    w = I.gen_weight(2, 0, I.SLOTS["w1"], 768, 3072, 0.02)
    assert abs(w.std() - 0.02) < 1e-4
    w_other = I.gen_weight(2, 1, I.SLOTS["w1"], 768, 3072, 0.02)
    c = np.corrcoef(w.reshape(-1)[:100000], w_other.reshape(-1)[:100000])[0, 1]
    assert abs(c) < 0.02
