"""Bit-identity of the forward pass at the configurations the acceptance gate
names: the same inputs give the same output bits on every CU quota, at every
batch size, and solo or co-located with another instance.

- a model whose FFN width (8384) is a multiple of 64 but of neither 96 nor
  128, the case where the GEMM's tile choice could once follow the quota into
  another K summation order;
- the BERT-base-shaped batch-32 forward across 64 / 128 / 192 / 256 CUs (the
  out-projection's tile changes with the quota at this batch);
- two BERT-base-shaped instances of batch 8, 200 back-to-back batches each at
  the quota pairs 64/192, 128/128 and 192/64, every batch equal to the solo run
  (the co-location configuration as specified), and the same at batch 32.

The outputs are compared as bit patterns (uint32 views of the fp32 logits)."""
import hashlib
import threading

import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from tests.gpu_util import DEV, compare, instance_config, run_instance

pytestmark = pytest.mark.gpu

QUOTAS = (64, 128, 192, 256)


def bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


def test_odd_ffn_width_is_bit_identical_across_quotas_and_batches():
    # d_model 2048, d_ff 8384 (= 131 * 64), 2 layers, causal pre-LN: FFN-up is
    # 8384 x 2048 (split K order), FFN-down 2048 x 8384
    # stress biases and LayerNorm affine; the Q and K std is scaled so that the
    # score std (d_model * qk_std^2) matches the stress init's at d_model 768
    # (2.8): at d_model 2048 qk_std 0.06 would give 7.4, a near one-hot softmax
    # whose ties the bf16 Q and K cannot resolve to the 2e-2 gate
    shape = W.model_shape("decoder_l24_d2048_s1024", n_layers=2, d_ff=8384, b_std=0.02, ln_std=0.02,
                          qk_std=0.0367)
    S = 128
    x = W.make_input(7100, 8, S, 2048)
    print("d_model 2048 / d_ff 8384: quotas and batch sizes", flush=True)
    with ie.Instance(**instance_config(shape, 8, S)) as inst:
        base = {}
        for q in QUOTAS:
            inst.set_quota(q)
            for B in (1, 8):
                got = run_instance(inst, x[:B])
                if B not in base:
                    base[B] = got
                assert np.array_equal(bits(got), bits(base[B])), (q, B)
        # sequence 0 alone equals sequence 0 of the batch of 8
        assert np.array_equal(bits(base[1][0]), bits(base[8][0]))
        inst.set_quota(256)
    ma, rl = compare(base[1], F.forward(x[:1], shape))
    print(f"  vs oracle: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert ma <= 2e-2 and rl <= 1e-2


def test_bert_base_batch32_bit_identical_across_quotas():
    shape = W.model_shape("bert_base_l12_d768_s128")
    x = W.make_input(2000 + 17, 32, 128, 768)
    print("bert B=32 across quotas", flush=True)
    with ie.Instance(**instance_config(shape, 32, 128)) as inst:
        ref = None
        for q in QUOTAS + (40,):
            inst.set_quota(q)
            got = run_instance(inst, x)
            if ref is None:
                ref = got
            assert np.array_equal(bits(got), bits(ref)), q


def _colocated_run(B, n_batches, pairs):
    shapes = [W.model_shape("bert_base_l12_d768_s128", seed=31), W.model_shape("bert_base_l12_d768_s128", seed=32)]
    insts = [ie.Instance(**instance_config(s, B, 128)) for s in shapes]
    try:
        xs = [[torch.from_numpy(W.make_input(31000 + 1000 * i + k, B, 128, 768)).to(DEV) for k in range(n_batches)]
              for i in range(2)]
        torch.cuda.synchronize()
        solo = []
        for i in range(2):
            insts[i].set_quota(256)
            hashes = []
            for k in range(n_batches):
                insts[i].submit(xs[i][k])
                hashes.append(hashlib.sha256(bits(insts[i].read_logits()).tobytes()).hexdigest())
            solo.append(hashes)
        for quotas in pairs:
            print(f"co-located B={B}: quotas {quotas}, {n_batches} batches each", flush=True)
            insts[0].set_quota(quotas[0], 0)
            insts[1].set_quota(quotas[1], quotas[0])
            got = [[None] * n_batches for _ in range(2)]
            errors = []
            start = threading.Barrier(2)

            def drive(i):
                try:
                    start.wait()
                    for k in range(n_batches):
                        insts[i].submit(xs[i][k])
                        got[i][k] = hashlib.sha256(bits(insts[i].read_logits()).tobytes()).hexdigest()
                except Exception as exc:   # surfaced below
                    errors.append(exc)

            threads = [threading.Thread(target=drive, args=(i,)) for i in range(2)]
            for t in threads:
                t.start()
            for t in threads:
                t.join(timeout=300)
            assert not errors, errors
            for i in range(2):
                bad = [k for k in range(n_batches) if got[i][k] != solo[i][k]]
                assert not bad, (quotas, i, bad[:5])
    finally:
        for inst in insts:
            inst.close()


def test_colocated_batch8_200_batches_equal_solo():
    _colocated_run(8, 200, ((64, 192), (128, 128), (192, 64)))


def test_colocated_batch32_equal_solo():
    _colocated_run(32, 20, ((64, 192), (128, 128), (192, 64)))
