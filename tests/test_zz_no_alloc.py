"""The allocation-free decode attention entry point against the allocating
one it is a variant of: the same kernels on the same inputs, so the contexts
must agree bit for bit; the first call also against the fp64 oracle.  Two
calls in a row, the second smaller than the first (the fixed scratch keeps the
first call's partial results, which the second must not read), then a size
beyond the scratch, which must be rejected before anything is launched."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
from oracle import forward as F
from tests.gpu_util import DEV, bf16_round, compare, f64, sync, to_dev

pytestmark = pytest.mark.gpu

NAN_BF16 = 0x7FC0


def _inputs(seed, B, H, n_keys, dh, k_rows, vt_stride):
    rng = np.random.default_rng(seed)
    q = bf16_round(rng.standard_normal((B, H, dh)))
    k = bf16_round(rng.standard_normal((B, H, k_rows, dh)))
    vt = bf16_round(rng.standard_normal((B, H, dh, vt_stride)))
    k.view(torch.int16)[:, :, n_keys:, :] = NAN_BF16      # cache positions past n_keys: arbitrary bits
    vt.view(torch.int16)[:, :, :, n_keys:] = NAN_BF16
    return q, k, vt


def _both(seed, B, H, n_keys, dh, k_rows, vt_stride):
    q, k, vt = _inputs(seed, B, H, n_keys, dh, k_rows, vt_stride)
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(vt)
    ref = torch.full((B, H * dh), float("nan"), dtype=torch.bfloat16, device=DEV)
    got = torch.full((B, H * dh), float("nan"), dtype=torch.bfloat16, device=DEV)
    ie.test_decode_attention(qd, kd, vd, ref, B, H, n_keys, dh, k_rows, vt_stride)
    ie.decode_attention_noalloc(qd, kd, vd, got, B, H, n_keys, dh, k_rows, vt_stride)
    sync()
    return q, k, vt, ref.cpu(), got.cpu()


def test_noalloc_equals_allocating_entry_point_twice():
    # first call: 12 chunks of 256 keys, 64 (batch, head) pairs, dh 128: 399 KB of partials
    print("no-alloc decode attention: B=4 H=16 keys=3000 dh=128", flush=True)
    q, k, vt, ref, got = _both(7, 4, 16, 3000, 128, 3100, 3008)
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
    B, H, n, dh = 4, 16, 3000, 128
    oracle = F.attention_context(f64(q)[:, :, None, :], f64(k)[:, :, :n], np.swapaxes(f64(vt)[..., :n], -1, -2),
                                 False).reshape(B, H * dh)
    ma, rl = compare(f64(got), oracle)
    print(f"  vs oracle: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert ma <= 2e-2 and rl <= 1e-2
    # second call, smaller: 5 chunks of 64 keys, 6 pairs, dh 64 (the scratch still
    # holds the first call's partials beyond what this call writes)
    print("no-alloc decode attention: B=2 H=3 keys=300 dh=64", flush=True)
    _, _, _, ref2, got2 = _both(8, 2, 3, 300, 64, 320, 320)
    assert torch.equal(got2.view(torch.int16), ref2.view(torch.int16))
    # and a single chunk, which writes the context directly
    _, _, _, ref3, got3 = _both(9, 1, 2, 40, 64, 40, 64)
    assert torch.equal(got3.view(torch.int16), ref3.view(torch.int16))


def test_noalloc_rejects_sizes_beyond_the_scratch():
    # 64 * 32 pairs, 32 chunks, dh 128: 2048 * 32 * 130 * 4 = 34 MB > 8 MiB -> EINVAL, nothing launched
    B, H, n, dh = 64, 32, 2048, 128
    t = torch.zeros(16, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ie.IefwdError) as e:
        ie.decode_attention_noalloc(t, t, t, t, B, H, n, dh, n, n)
    assert e.value.status == ie.EINVAL
    assert "scratch" in str(e.value)
