"""Training steps on the GPU (iefwd_train_*) against the fp64 training oracle:
the loss, every parameter's gradient, the AdamW update and moments, and the
logits; determinism across quotas; the error paths."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from oracle import train as T
from tests.gpu_util import DEV, instance_config

pytestmark = pytest.mark.gpu

SMALL = dict(W.STRESS_INIT, n_layers=2, d_model=128, n_heads=2, d_ff=256, pre_ln=0, causal=0, n_out=3)
SLOTS = {"wqkv": 0, "bqkv": 1, "wo": 2, "bo": 3, "ln1_g": 4, "ln1_b": 5, "w1": 6, "b1": 7, "w2": 8, "b2": 9,
         "ln2_g": 10, "ln2_b": 11}
# per-tensor gradient gate: relative L2 error against the fp64 oracle.  The
# GPU keeps bf16 activations and bf16 backward operands (2^-9 relative
# rounding each) with fp32 accumulation; through a two-layer stack that
# leaves about 1e-2 relative error in a gradient tensor.
GRAD_REL_L2 = 3e-2
LOSS_REL = 5e-3


def shape_of(over):
    return W.model_shape("encoder_l1_d128_s32_b2", **over)


def rel_l2(a, b):
    return float(np.linalg.norm(np.asarray(a, np.float64) - b) / max(np.linalg.norm(b), 1e-30))


def oracle_tensors(tree, shape):
    """(layer, slot, name, fp64 array) for every parameter of an oracle tree."""
    out = []
    for l, w in enumerate(tree["layers"]):
        for k, slot in SLOTS.items():
            out.append((l, slot, f"layer{l}.{k}", w[k]))
    out.append((shape["n_layers"], 14, "wh", tree["wh"]))
    out.append((shape["n_layers"], 15, "bh", tree["bh"]))
    return out


def make_batch(shape, B, S, seed):
    x = W.make_input(seed, B, S, shape["d_model"])
    labels = W.make_labels(seed + 1, B, S, shape["n_out"])
    return x, labels


@pytest.mark.parametrize("causal,B,S", [(0, 2, 32), (1, 1, 64), (0, 4, 48)])
def test_one_step_matches_oracle(causal, B, S):
    shape = shape_of(dict(SMALL, causal=causal))
    print(f"train step causal={causal} B={B} S={S}", flush=True)
    x, labels = make_batch(shape, B, S, 300 + S)
    params = T.initial_params(shape)
    loss_ref, grads_ref, _ = T.loss_and_grads(params, x, labels, shape)
    with ie.Trainer(**instance_config(shape, B, S)) as tr:
        tr.step(x, labels)
        loss = tr.loss()
        logits = tr.read_logits()
        print(f"  loss gpu {loss:.6f} oracle {loss_ref:.6f}", flush=True)
        assert abs(loss - loss_ref) <= LOSS_REL * abs(loss_ref)
        ref_logits = F.forward(x, shape)
        assert np.max(np.abs(logits - ref_logits)) <= 2e-2 and rel_l2(logits, ref_logits) <= 1e-2
        worst = 0.0
        for layer, slot, name, ref in oracle_tensors(grads_ref, shape):
            g = tr.export(layer, slot, ie.TRAIN_GRAD, ref.shape)
            e = rel_l2(g, ref)
            worst = max(worst, e)
            assert np.all(np.isfinite(g)), name
            assert e <= GRAD_REL_L2, (name, e)
        print(f"  worst gradient rel-L2 {worst:.3e}", flush=True)

        # the update: the oracle's AdamW applied to the GPU's own gradients, with
        # the hyper-parameters the library holds (their fp32 values)
        hp = {k: float(np.float32(v)) for k, v in T.ADAMW_DEFAULTS.items()}
        for layer, slot, name, w0 in oracle_tensors(params, shape):
            g = tr.export(layer, slot, ie.TRAIN_GRAD, w0.shape).astype(np.float64)
            key = name.split(".")[-1]
            w1, m1, v1 = T.adamw_update(w0, g, np.zeros_like(w0), np.zeros_like(w0), 1, key in T.DECAYED, **hp)
            got_w = tr.export(layer, slot, ie.TRAIN_MASTER, w0.shape)
            got_m = tr.export(layer, slot, ie.TRAIN_MOMENT1, w0.shape)
            got_v = tr.export(layer, slot, ie.TRAIN_MOMENT2, w0.shape)
            # fp32 update arithmetic: a few ulps of w and of the step lr
            assert np.all(np.abs(got_w - w1) <= 4e-7 * np.abs(w1) + 4 * 2 ** -24 * hp["lr"] + 1e-12), name
            assert np.all(np.abs(got_m - m1) <= 2e-7 * np.abs(m1) + 1e-30), name
            assert np.all(np.abs(got_v - v1) <= 2e-7 * np.abs(v1) + 1e-30), name
        assert tr.steps() == 1


@pytest.mark.parametrize("d", [512, 1024, 2048])
def test_one_step_wide_models(d):
    """One layer at widths that take the other LayerNorm-backward forms (d 512
    and 1024: 2 and 4 column vectors per lane; d 2048: the two-kernel form)."""
    shape = shape_of(dict(SMALL, n_layers=1, d_model=d, n_heads=d // 64, d_ff=2 * d))
    print(f"train step d={d}", flush=True)
    x, labels = make_batch(shape, 1, 64, 500 + d)
    params = T.initial_params(shape)
    loss_ref, grads_ref, _ = T.loss_and_grads(params, x, labels, shape)
    with ie.Trainer(**instance_config(shape, 1, 64)) as tr:
        tr.step(x, labels)
        assert abs(tr.loss() - loss_ref) <= LOSS_REL * abs(loss_ref)
        for layer, slot, name, ref in oracle_tensors(grads_ref, shape):
            g = tr.export(layer, slot, ie.TRAIN_GRAD, ref.shape)
            e = rel_l2(g, ref)
            assert np.all(np.isfinite(g)), name
            assert e <= GRAD_REL_L2, (name, e)


def test_steps_deterministic_across_quotas():
    shape = shape_of(SMALL)
    x, labels = make_batch(shape, 2, 32, 77)
    results = []
    for quota in (256, 64):
        with ie.Trainer(**instance_config(shape, 2, 32)) as tr:
            tr.set_quota(quota)
            xd = torch.from_numpy(x).to(DEV)
            ld = torch.from_numpy(labels).to(DEV)
            losses = []
            for _ in range(3):
                tr.step(xd, ld)
                losses.append(tr.loss())
            w = tr.export(0, 0, ie.TRAIN_MASTER, (shape["d_model"], 3 * shape["d_model"]))
            results.append((losses, w))
    assert results[0][0] == results[1][0]
    assert np.array_equal(results[0][1].view(np.uint32), results[1][1].view(np.uint32))


def test_training_reduces_the_loss_like_the_oracle():
    shape = shape_of(dict(SMALL, n_layers=1))
    x, labels = make_batch(shape, 2, 32, 91)
    hp = dict(lr=2e-3, weight_decay=0.0)
    params = T.initial_params(shape)
    opt = T.AdamW(params, **hp)
    ref = [T.train_step(params, opt, x, labels, shape) for _ in range(5)]
    with ie.Trainer(train=hp, **instance_config(shape, 2, 32)) as tr:
        got = []
        for _ in range(25):
            tr.step(x, labels)
            got.append(tr.loss())
    print("  gpu", [round(v, 5) for v in got[:5]], "oracle", [round(v, 5) for v in ref], flush=True)
    for a, b in zip(got[:5], ref):
        assert abs(a - b) <= 2e-2 * abs(b)
    assert got[-1] < 0.7 * got[0]


def test_train_errors():
    shape = shape_of(SMALL)
    with pytest.raises(ie.IefwdError) as e:
        ie.Trainer(**instance_config(dict(shape, pre_ln=1), 2, 32))
    assert e.value.status == ie.EINVAL
    with pytest.raises(ie.IefwdError) as e:
        ie.Trainer(**instance_config(shape, 2, 256))          # max_seq > 128
    assert e.value.status == ie.EINVAL
    with pytest.raises(ie.IefwdError) as e:
        ie.Trainer(train=dict(beta1=1.0), **instance_config(shape, 2, 32))
    assert e.value.status == ie.EINVAL
    x, labels = make_batch(shape, 2, 32, 5)
    with ie.Trainer(**instance_config(shape, 2, 32)) as tr:
        with pytest.raises(ie.IefwdError) as e:
            tr.loss()                                          # no step yet
        assert e.value.status == ie.ESTATE
        with pytest.raises(ie.IefwdError) as e:
            tr.step(x[:, :31], labels[:, :31])                 # 62 tokens: not a multiple of 64
        assert e.value.status == ie.EINVAL
        with pytest.raises(ie.IefwdError) as e:
            tr.export(0, 12, ie.TRAIN_GRAD, (128,))
        assert e.value.status == ie.EINVAL
    with ie.Instance(**instance_config(shape, 2, 32)) as inst:   # an inference instance
        st = ie.lib().iefwd_train_step(inst._h, x.ctypes.data, labels.ctypes.data, 2, 32, 0)
        assert st == ie.ESTATE


def test_bert_base_sized_step():
    """The BERT-base-shaped model (12 layers, d 768, 12 heads, F 3072) at
    batch 2, seq 128: loss and a sample of gradients against the oracle."""
    shape = W.model_shape("bert_base_l12_d768_s128")
    B, S = 2, 128
    print("bert-base train step", flush=True)
    x, labels = make_batch(shape, B, S, 2024)
    params = T.initial_params(shape)
    loss_ref, grads_ref, _ = T.loss_and_grads(params, x, labels, shape)
    with ie.Trainer(**instance_config(shape, B, S)) as tr:
        tr.step(x, labels)
        loss = tr.loss()
        print(f"  loss gpu {loss:.6f} oracle {loss_ref:.6f}", flush=True)
        assert abs(loss - loss_ref) <= LOSS_REL * abs(loss_ref)
        for layer, slot, name, ref in oracle_tensors(grads_ref, shape):
            if layer not in (0, 11, 12):
                continue
            g = tr.export(layer, slot, ie.TRAIN_GRAD, ref.shape)
            e = rel_l2(g, ref)
            print(f"  {name}: rel-L2 {e:.3e}", flush=True)
            assert e <= 2 * GRAD_REL_L2, (name, e)
