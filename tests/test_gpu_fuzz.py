"""Seeded random shapes for the kernels' parity tests: each case runs the
same check as the hand-picked cases (the fp64 oracle and its error bounds),
at sizes drawn from the kernels' documented limits, so tile edges, ragged
tails, K-group choices and chunk counts are hit in combinations nobody chose."""
import numpy as np
import pytest

import paper_2503_05130_amd as ie
from tests.test_gpu_decode import test_decode_attention_kernel as _decode_attention_case
from tests.test_gpu_decode import test_gemm_skinny as _skinny_case
from tests.test_gpu_kernels import test_attention as _attention_case
from tests.test_gpu_kernels import test_gemm_epilogues as _gemm_case
from tests.test_gpu_kernels import test_layernorm as _layernorm_case

pytestmark = pytest.mark.gpu

_rng = np.random.default_rng(20250305)
EPIS = (ie.EPI_BIAS_BF16, ie.EPI_BIAS_GELU_BF16, ie.EPI_BIAS_RESID_F32)


def _gemm_cases(n):
    out = []
    while len(out) < n:
        M = int(_rng.integers(1, 2049))
        N = 64 * int(_rng.integers(1, 25))
        K = 64 * int(_rng.integers(1, 49))
        if M * N * K <= 1.2e9:                 # the fp64 reference stays around a second
            out.append((M, N, K, int(_rng.choice(EPIS))))
    return out


def _attention_cases(n):
    return [(int(_rng.integers(1, 4)), int(_rng.integers(1, 4)), int(_rng.integers(1, 700)),
             int(_rng.choice((64, 128))), bool(_rng.integers(0, 2)), float(_rng.choice((0.5, 1.0, 2.0))))
            for _ in range(n)]


def _layernorm_cases(n):
    return [(int(_rng.integers(1, 700)), 128 * int(_rng.integers(1, 33))) for _ in range(n)]


def _decode_cases(n):
    out = []
    for _ in range(n):
        n_keys = int(_rng.integers(1, 4097))
        k_rows = n_keys + int(_rng.integers(0, 64))
        vt_stride = (n_keys + 63) // 64 * 64 + 64 * int(_rng.integers(0, 2))
        out.append((int(_rng.integers(1, 4)), int(_rng.integers(1, 5)), n_keys, int(_rng.choice((64, 128))),
                    k_rows, vt_stride))
    return out


def _skinny_cases(n):
    out = []
    while len(out) < n:
        M = int(_rng.integers(1, 17))
        N = 16 * int(_rng.integers(1, 257))
        K = 32 * int(_rng.integers(1, 129))
        ln = bool(_rng.integers(0, 2)) and K <= 4096 and M * K <= 16384
        if M * N * K <= 2e8:
            out.append((M, N, K, int(_rng.choice(EPIS)), ln))
    return out


@pytest.mark.parametrize("M,N,K,epi", _gemm_cases(40))
def test_gemm_random(M, N, K, epi):
    _gemm_case(M, N, K, epi)


@pytest.mark.parametrize("B,H,S,dh,causal,scale", _attention_cases(20))
def test_attention_random(B, H, S, dh, causal, scale):
    _attention_case(B, H, S, dh, causal, scale)


@pytest.mark.parametrize("rows,d", _layernorm_cases(12))
def test_layernorm_random(rows, d):
    _layernorm_case(rows, d)


@pytest.mark.parametrize("B,H,n_keys,dh,k_rows,vt_stride", _decode_cases(16))
def test_decode_attention_random(B, H, n_keys, dh, k_rows, vt_stride):
    _decode_attention_case(B, H, n_keys, dh, k_rows, vt_stride)


@pytest.mark.parametrize("M,N,K,epi,ln", _skinny_cases(20))
def test_gemm_skinny_random(M, N, K, epi, ln):
    _skinny_case(M, N, K, epi, ln)
