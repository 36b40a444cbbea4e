"""The decode-step product reading the packed copy of its weights: the copy is
the layout the header defines, and the product on it equals the product on
the row-major weights bit for bit (only the addresses of the loads differ)."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
from tests.gpu_util import DEV, bf16_round, sync, to_dev

pytestmark = pytest.mark.gpu


def packed_reference(w_nk, groups):
    """The packed layout written out from its definition: 16-byte piece
    i = (b * steps + s) * 64 + l holds W[f, k .. k + 7] with r = l % 16,
    c = l // 16, f = b * (16 / groups) + r % (16 / groups),
    k = (r // (16 / groups)) * (K / groups) + 32 s + 8 c."""
    N, K = w_nk.shape
    fpw, kg = 16 // groups, K // groups
    steps = kg // 32
    out = np.empty((N // fpw, steps, 64, 8), dtype=w_nk.dtype)
    for l in range(64):
        r, c = l % 16, l // 16
        f = np.arange(N // fpw) * fpw + r % fpw
        for s in range(steps):
            k = (r // fpw) * kg + 32 * s + 8 * c
            out[:, s, l, :] = w_nk[f, k:k + 8]
    return out.reshape(-1)


@pytest.mark.parametrize("N,K,groups", [(16, 32, 1), (64, 256, 2), (128, 512, 4), (48, 96, 1), (32, 2048, 4)])
def test_pack_layout(N, K, groups):
    print(f"pack N={N} K={K} groups={groups}", flush=True)
    rng = np.random.default_rng(N + K + groups)
    bits = rng.integers(0, 1 << 16, size=(N, K), dtype=np.uint16)
    w = torch.from_numpy(bits.view(np.int16)).to(DEV)
    dst = torch.empty(N * K, dtype=torch.int16, device=DEV)
    ie.test_skinny_pack(w, dst, N, K, groups)
    sync()
    got = dst.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, packed_reference(bits, groups))


# M, N, K, epilogue, LayerNorm activations: the decoder's products at d 2048 and smaller ones
PACKED = [
    (1, 6144, 2048, ie.EPI_BIAS_BF16, True),        # QKV with the fused LayerNorm
    (2, 6144, 2048, ie.EPI_BIAS_BF16, True),
    (4, 8192, 2048, ie.EPI_BIAS_GELU_BF16, True),   # FFN-up
    (2, 2048, 2048, ie.EPI_BIAS_RESID_F32, False),  # out-projection: 4 K-groups
    (3, 2048, 8192, ie.EPI_BIAS_RESID_F32, False),  # FFN-down: 4 K-groups
    (8, 1024, 2048, ie.EPI_BIAS_BF16, False),       # 2 K-groups
    (16, 768, 96, ie.EPI_BIAS_GELU_BF16, False),    # 1 K-group, fewer K steps than waves
    (3, 2304, 768, ie.EPI_BIAS_GELU_BF16, True),    # 2 K-groups with the prologue
]


@pytest.mark.parametrize("M,N,K,epi,ln", PACKED)
def test_packed_product_bit_identical(M, N, K, epi, ln):
    g = ie.test_skinny_groups(M, N, K, ln)
    print(f"packed skinny M={M} N={N} K={K} epi={epi} ln={ln} groups={g}", flush=True)
    rng = np.random.default_rng(M * 7 + N + K + epi)
    w = to_dev(bf16_round(rng.standard_normal((N, K)) * 0.05))
    bias = to_dev(bf16_round(rng.standard_normal(N) * 0.1))
    resid = torch.from_numpy(rng.standard_normal((M, N)).astype(np.float32)).to(DEV)
    r_d = resid if epi == ie.EPI_BIAS_RESID_F32 else None
    odt = torch.float32 if epi == ie.EPI_BIAS_RESID_F32 else torch.bfloat16
    if ln:
        z = torch.from_numpy((rng.standard_normal((M, K)) * 2.0 + 0.5).astype(np.float32)).to(DEV)
        gam = torch.from_numpy((1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32)).to(DEV)
        bet = torch.from_numpy((0.1 * rng.standard_normal(K)).astype(np.float32)).to(DEV)
        lnarg, a = (z, gam, bet, 1e-5), None
    else:
        lnarg, a = None, to_dev(bf16_round(rng.standard_normal((M, K))))
    packed = torch.empty(N * K, dtype=torch.bfloat16, device=DEV)
    ie.test_skinny_pack(w, packed, N, K, g)
    ref = torch.full((M, N), float("nan"), dtype=odt, device=DEV)
    got = torch.full((M, N), float("nan"), dtype=odt, device=DEV)
    ie.test_gemm_skinny(epi, a, w, bias, r_d, ref, M, N, K, ln=lnarg)
    for _ in range(2):                               # twice: no state carried between calls
        ie.test_gemm_skinny_packed(epi, a, packed, g, bias, r_d, got, M, N, K, ln=lnarg)
        sync()
        assert torch.equal(got.view(torch.int16 if odt == torch.bfloat16 else torch.int32),
                           ref.view(torch.int16 if odt == torch.bfloat16 else torch.int32))
        got.fill_(float("nan"))


def test_packed_product_rejects_other_group_count():
    N, K = 2048, 2048
    w = torch.zeros((N, K), dtype=torch.bfloat16, device=DEV)
    b = torch.zeros(N, dtype=torch.bfloat16, device=DEV)
    a = torch.zeros((8, K), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros((8, N), dtype=torch.bfloat16, device=DEV)
    packed = torch.empty(N * K, dtype=torch.bfloat16, device=DEV)
    assert ie.test_skinny_groups(2, N, K, False) == 4 and ie.test_skinny_groups(8, N, K, False) == 2
    ie.test_skinny_pack(w, packed, N, K, 4)
    with pytest.raises(ie.IefwdError) as e:            # 8 rows use 2 K-groups
        ie.test_gemm_skinny_packed(ie.EPI_BIAS_BF16, a, packed, 4, b, None, out, 8, N, K)
    assert e.value.status == ie.EINVAL
    for bad in ((w, packed, N, K, 3), (w, packed, N, 48, 1), (w, packed, 40, K, 1)):
        with pytest.raises(ie.IefwdError) as e:
            ie.test_skinny_pack(*bad)
        assert e.value.status == ie.EINVAL
