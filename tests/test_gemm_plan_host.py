"""Host checks of the GEMM launch plan (no GPU needed): the K summation order
of a product is a function of the weight shape (N, K) alone, and the tile the
library picks always sums in that order, whatever the batch (M), the CU
quota or the width the tiles must divide.  This is what makes an output
element's bits independent of the quota and of the other rows in the batch."""
import itertools

import pytest

import paper_2503_05130_amd as ie

MS = [1, 2, 7, 16, 64, 100, 128, 256, 512, 1000, 2048, 4096, 8192, 16384]
N_CUS = [8, 16, 32, 64, 96, 128, 160, 192, 224, 256]
KS = [64, 128, 768, 1024, 1984, 2048, 2112, 3072, 4096, 8192, 8384, 16384]
# widths (features) of the products of every model the library accepts: 3d, d, d_ff; plus the
# widths that are multiples of 64 but of neither 96 nor 128 (d_ff = 8384, 320, 704, ...)
NS = [64, 128, 192, 320, 384, 704, 768, 1024, 1088, 2304, 3072, 4096, 6144, 8192, 8384, 12288, 16448]


def _plan(M, N, K, align, n_cu):
    return ie.test_gemm_plan(M, N, K, align, n_cu)


def test_k_order_depends_on_weight_shape_only():
    for N, K in itertools.product(NS, KS):
        orders = set()
        for M, n_cu in itertools.product(MS, N_CUS):
            k_order, tile_order, bm, bn = _plan(M, N, K, N, n_cu)
            assert tile_order == k_order, (M, N, K, n_cu, bm, bn)
            assert N % bn == 0 and bm > 0
            orders.add(k_order)
        assert len(orders) == 1, (N, K, orders)
        assert orders == {1 if K >= 2048 else 0}


@pytest.mark.parametrize("d", [128, 256, 768, 1024, 2048, 4096])
def test_qkv_tiles_do_not_straddle_q_k_v(d):
    # the QKV product's tiles divide d_model, so no tile mixes Q, K and V columns
    for M, n_cu in itertools.product(MS, N_CUS):
        k_order, tile_order, bm, bn = _plan(M, 3 * d, d, d, n_cu)
        assert d % bn == 0 and tile_order == k_order


def test_the_width_that_once_broke_the_order():
    # d_model 2048 with d_ff 8384: FFN-up N = 8384, K = 2048 (split order), at
    # every batch and quota; before the fix 64-128 CUs took a sequential tile
    for M in (128, 1024, 8192):
        for n_cu in (64, 128, 192, 256):
            assert _plan(M, 8384, 2048, 8384, n_cu)[:2] == (1, 1)


def test_plan_rejects_bad_arguments():
    for args in [(0, 64, 64, 64, 256), (1, 96, 64, 96, 256), (1, 64, 96, 64, 256), (1, 128, 64, 96, 256),
                 (1, 128, 64, 128, 0)]:
        with pytest.raises(ie.IefwdError) as e:
            _plan(*args)
        assert e.value.status == ie.EINVAL


@pytest.mark.parametrize("M,N,K,ln,groups", [
    (2, 6144, 2048, True, 1),     # d-2048 QKV with the LayerNorm prologue: 2 groups would need 768 workgroups
    (2, 6144, 2048, False, 2),
    (4, 8192, 2048, True, 1),     # FFN-up
    (2, 2048, 2048, False, 4),    # out-projection
    (4, 2048, 8192, False, 4),    # FFN-down: up to 4 rows take 4 groups
    (8, 2048, 8192, False, 2),    # 5-8 rows: 2
    (9, 2048, 8192, False, 1),    # 9-16 rows: 1
    (3, 2304, 768, True, 2),      # 4 groups would need 576 workgroups, past 2 per CU
    (2, 2048, 96, False, 1),      # K not a multiple of 64
])
def test_skinny_group_count(M, N, K, ln, groups):
    """The decode product's K-group rule: the most groups (up to 4, at most 16 /
    groups rows) whose N / (16 / groups) workgroups fit 3 per CU (2 with the
    LayerNorm prologue) on 256 CUs; the packed weight copy is made for it."""
    assert ie.test_skinny_groups(M, N, K, ln) == groups


@pytest.mark.parametrize("M,N,K,n_cu,tile", [
    # BERT-base batch 32 (4096 tokens): FFN-down (even/odd order), FFN-up, out-projection
    (4096, 768, 3072, 256, (64, 96)),    # 512 tiles, two per CU
    (4096, 768, 3072, 192, (128, 128)),  # 64 x 96 would leave some CUs three tiles
    (4096, 768, 3072, 128, (64, 96)),    # four per CU either way: the first choice stays
    (4096, 3072, 768, 256, (128, 192)),
    (4096, 3072, 768, 192, (128, 128)),
    (4096, 768, 768, 256, (128, 96)),
    (4096, 768, 768, 192, (128, 128)),
    (4096, 2304, 768, 192, (128, 192)),  # QKV: 384 tiles fill 192 CUs twice
])
def test_tile_balances_the_share(M, N, K, n_cu, tile):
    """On shares whose CU count leaves the first-choice tiles unevenly spread, a
    128 x 128 tile of the same K order is taken when it leaves the busiest CU
    with at most 90% of the work."""
    k_order, tile_order, bm, bn = ie.test_gemm_plan(M, N, K, N, n_cu)
    assert (bm, bn) == tile and k_order == tile_order


@pytest.mark.parametrize("n_cu,plain,ln_residual", [
    (64, (128, 192), (128, 128)),    # the 128 x 192 tile would spill with the LayerNorm residual
    (128, (128, 96), (128, 96)),
    (256, (128, 96), (128, 96)),
])
def test_ln_residual_epilogue_skips_the_widest_tile(n_cu, plain, ln_residual):
    for flag, want in ((False, plain), (True, ln_residual)):
        k_order, tile_order, bm, bn = ie.test_gemm_plan(4096, 768, 768, 768, n_cu, flag)
        assert (bm, bn) == want and k_order == tile_order == 0
