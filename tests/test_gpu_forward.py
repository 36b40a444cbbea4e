"""End-to-end parity of the forward pass (C ABI -> HIP kernels) against the fp64
oracle, plus the determinism properties of the quota layer: bit-identical
outputs across CU quotas, repeats, batch composition and co-location.

Acceptance for logits / hidden states: max-abs <= 2e-2 and rel-L2 <= 1e-2 over
the whole output of each compared batch (or of each sampled sequence)."""
import threading

import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from oracle import init_spec as I
from tests.gpu_util import DEV, compare, instance_config, run_instance

pytestmark = pytest.mark.gpu

MAX_ABS, REL_L2 = 2e-2, 1e-2


def check(got, ref, what=""):
    ma, rl = compare(got, ref)
    print(f"  {what}: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert np.all(np.isfinite(got))
    assert ma <= MAX_ABS and rl <= REL_L2, (what, ma, rl)


# ------------------------------------------------------------------------ small shapes, full oracle
SMALL = [
    # name, shape overrides, batch, seq
    ("encoder_l1_d128_s32_b2", {}, 2, 32),
    ("encoder_l1_d128_s32_b2", dict(n_out=2), 2, 32),
    ("encoder_l1_d128_s32_b2", W.STRESS_INIT, 2, 32),
    ("encoder_l1_d128_s32_b2", dict(W.STRESS_INIT, n_layers=3, causal=1), 3, 37),
    ("encoder_l1_d128_s32_b2", dict(W.STRESS_INIT, pre_ln=1, causal=1, n_out=3), 2, 45),
    ("encoder_l1_d128_s32_b2", dict(W.STRESS_INIT, d_model=256, n_heads=2, d_ff=640, n_layers=2), 3, 19),
    ("encoder_l1_d128_s32_b2", dict(W.STRESS_INIT, d_model=384, n_heads=6, d_ff=1536, n_layers=2, pre_ln=1), 2, 130),
    ("encoder_l1_d128_s32_b2", dict(d_model=128, n_heads=2, d_ff=512, n_layers=2, pre_ln=1, causal=1), 1, 1),
]


@pytest.mark.parametrize("name,over,batch,seq", SMALL)
def test_small_forward_matches_oracle(name, over, batch, seq):
    shape = W.model_shape(name, **over)
    print(f"forward {name} {over} B={batch} S={seq}", flush=True)
    x = W.make_input(W.WORKLOADS[name]["input_seed"] + seq, batch, seq, shape["d_model"])
    with ie.Instance(**instance_config(shape, max_batch=batch + 1, max_seq=seq + 5)) as inst:
        got = run_instance(inst, x)
    check(got, F.forward(x, shape), "small")


def test_weights_equal_oracle_init_spec():
    # T2: the library's host-generated weights equal the oracle's, bit for bit
    shape = W.model_shape("encoder_l1_d128_s32_b2", **W.STRESS_INIT, n_layers=2, n_out=3)
    with ie.Instance(**instance_config(shape, 2, 32)) as inst:
        for layer in range(2):
            ref = I.layer_weights(shape, layer)
            for slot_name, slot in I.SLOTS.items():
                if slot >= 12:
                    continue
                got = inst.export_tensor(layer, slot)
                want = ref[slot_name]
                if got.dtype == np.uint16:
                    got = I.bf16_bits_to_f64(got)
                assert np.array_equal(got.astype(np.float64), want.reshape(got.shape)), (layer, slot_name)
        g = I.global_weights(shape)
        for slot_name in ("lnf_g", "lnf_b", "wh", "bh"):
            got = inst.export_tensor(shape["n_layers"], I.SLOTS[slot_name])
            if got.dtype == np.uint16:
                got = I.bf16_bits_to_f64(got)
            assert np.array_equal(got.astype(np.float64), g[slot_name].reshape(got.shape)), slot_name


# ------------------------------------------------------------------------ BERT-base-shaped stack
def bert_x(batch, k=0):
    w = W.WORKLOADS["bert_base_l12_d768_s128"]
    return W.make_input(w["input_seed"] + k, batch, w["seq"], 768)


@pytest.fixture(scope="module")
def bert():
    shape = W.model_shape("bert_base_l12_d768_s128")
    inst = ie.Instance(**instance_config(shape, max_batch=32, max_seq=128))
    yield shape, inst
    inst.close()


@pytest.mark.parametrize("batch", [1, 8, 32])
def test_bert_base_matches_oracle(bert, batch):
    shape, inst = bert
    print(f"bert B={batch}", flush=True)
    x = bert_x(batch)
    got = run_instance(inst, x)
    # sequences are independent: check the first and last sequence of the batch
    for b in sorted({0, batch - 1}):
        check(got[b:b + 1], F.forward(x[b:b + 1], shape), f"seq {b}")


def test_bert_base_post_ln_hidden_state_invariant():
    # n_out = 0: every output row of a post-LN stack (gamma = 1, beta = 0) has mean 0, var 1
    shape = W.model_shape("bert_base_l12_d768_s128", n_out=0)
    with ie.Instance(**instance_config(shape, 32, 128)) as inst:
        got = run_instance(inst, bert_x(32, k=5)).astype(np.float64)
    assert np.max(np.abs(got.mean(-1))) < 1e-5
    assert np.max(np.abs(got.var(-1) - 1.0)) < 1e-3


def test_bit_identical_across_quotas_and_repeats(bert):
    shape, inst = bert
    x = bert_x(8, k=1)
    inst.set_quota(256)
    base = run_instance(inst, x)
    for q in (8, 64, 128, 192, 256, 40):
        inst.set_quota(q)
        got = run_instance(inst, x)
        assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), q
        n_set = sum(bin(w).count("1") for w in inst.get_cu_mask())
        assert n_set == q
    inst.set_quota(256)


def test_batch_invariance(bert):
    # a sequence's logits do not depend on the other sequences in its batch
    shape, inst = bert
    x = bert_x(8, k=2)
    full = run_instance(inst, x)
    for b in (0, 5):
        alone = run_instance(inst, x[b:b + 1])
        assert np.array_equal(alone[0].view(np.uint32), full[b].view(np.uint32))


def test_host_and_device_inputs_agree(bert):
    shape, inst = bert
    x = bert_x(2, k=3)
    inst.submit(x)                       # host buffer, copied before submit returns
    host = inst.read_logits()
    dev = run_instance(inst, x)
    assert np.array_equal(host.view(np.uint32), dev.view(np.uint32))
    out_dev = torch.empty((2, 128, 2), dtype=torch.float32, device=DEV)
    xd = torch.from_numpy(x).to(DEV)
    inst.submit(xd)
    inst.read_logits(out_dev)
    assert np.array_equal(out_dev.cpu().numpy().view(np.uint32), host.view(np.uint32))


def test_state_errors(bert):
    shape, inst = bert
    x = torch.from_numpy(bert_x(1, k=4)).to(DEV)
    inst.submit(x)
    with pytest.raises(ie.IefwdError) as e:
        inst.submit(x)                   # one batch in flight per instance
    assert e.value.status == ie.ESTATE
    inst.wait()
    assert inst.last_batch_ms() > 0
    with pytest.raises(ie.IefwdError) as e:
        inst.read_logits(np.empty((1, 128, 3), np.float32))      # wrong size
    assert e.value.status == ie.EINVAL
    for b, s in ((0, 128), (33, 128), (1, 129), (1, 0)):
        assert ie.lib().iefwd_submit(inst._h, x.data_ptr(), b, s, 1) == ie.EINVAL
    assert ie.lib().iefwd_submit(inst._h, None, 1, 128, 1) == ie.EINVAL
    with pytest.raises(ie.IefwdError):
        inst.set_quota(0)
    with pytest.raises(ie.IefwdError):
        inst.set_quota(10 ** 6)


def test_fresh_instance_read_before_submit():
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    with ie.Instance(**instance_config(shape, 2, 32)) as inst:
        with pytest.raises(ie.IefwdError) as e:
            inst.read_logits(np.empty((2, 32, 128), np.float32))
        assert e.value.status == ie.ESTATE
        with pytest.raises(ie.IefwdError) as e:
            inst.last_batch_ms()
        assert e.value.status == ie.ESTATE


def test_colocated_equals_solo():
    # two BERT-base-shaped instances (independent seeds) co-located on disjoint
    # CUs (128/128, 64/192) and on the same CUs (128 each, both at bit 0),
    # driven from two host threads: every batch equals the solo full-quota
    # result bit for bit
    n_batches = 12
    shapes = [W.model_shape("bert_base_l12_d768_s128", seed=31), W.model_shape("bert_base_l12_d768_s128", seed=32)]
    xs = [[W.make_input(31000 + 1000 * i + k, 8, 128, 768) for k in range(n_batches)] for i in range(2)]
    insts = [ie.Instance(**instance_config(s, 8, 128)) for s in shapes]
    try:
        solo = [[run_instance(insts[i], xs[i][k]) for k in range(n_batches)] for i in range(2)]
        for quotas in (((128, 0), (128, 128)), ((64, 0), (192, 64)), ((128, 0), (128, 0))):
            for inst, (q, first) in zip(insts, quotas):
                inst.set_quota(q, first)
            results = [[None] * n_batches for _ in range(2)]
            errors = []

            def drive(i):
                try:
                    dx = [torch.from_numpy(x).to(DEV) for x in xs[i]]
                    torch.cuda.synchronize()
                    for k in range(n_batches):
                        insts[i].submit(dx[k])
                        results[i][k] = insts[i].read_logits()
                except Exception as exc:   # surfaced below
                    errors.append(exc)

            threads = [threading.Thread(target=drive, args=(i,)) for i in range(2)]
            for t in threads:
                t.start()
            for t in threads:
                t.join(timeout=120)
            assert not errors, errors
            for i in range(2):
                for k in range(n_batches):
                    assert np.array_equal(results[i][k].view(np.uint32), solo[i][k].view(np.uint32)), (quotas, i, k)
    finally:
        for inst in insts:
            inst.close()


# ------------------------------------------------------------------------ causal decoders, full size
@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,prefix", [("decoder_l24_d1024_s512", 64), ("decoder_l24_d2048_s1024", 32)])
def test_decoder_full_sequence_matches_oracle(name, prefix):
    # the full-size batch on the GPU; the oracle runs the first sequence at its
    # full length (every position, so every key chunk of the online softmax and
    # every query workgroup), and the last sequence on a prefix (causal: outputs
    # at positions < p depend only on tokens < p)
    w = W.WORKLOADS[name]
    shape = W.model_shape(name)
    B, S = w["batch"], w["seq"]
    print(f"decoder {name} B={B} S={S}: sequence 0 whole, sequence {B - 1} prefix {prefix}", flush=True)
    x = W.make_input(w["input_seed"], B, S, shape["d_model"])
    with ie.Instance(**instance_config(shape, B, S)) as inst:
        got = run_instance(inst, x)
    assert np.all(np.isfinite(got))
    check(got[B - 1:B, :prefix], F.forward(x[B - 1:B, :prefix], shape), f"seq {B - 1} prefix")
    check(got[0:1], F.forward(x[0:1], shape), "seq 0 whole")


@pytest.mark.timeout(600)
def test_bert_base_batch32_stress_init_matches_oracle():
    # stress init (biases, LN affine, peaked attention) at the headline batch:
    # 8 sequences spread over the batch against the oracle
    shape = W.model_shape("bert_base_l12_d768_s128", **W.STRESS_INIT)
    x = bert_x(32, k=9)
    print("bert B=32 stress init", flush=True)
    with ie.Instance(**instance_config(shape, 32, 128)) as inst:
        got = run_instance(inst, x)
    idx = [0, 5, 9, 14, 18, 23, 27, 31]
    check(got[idx], F.forward(x[idx], shape), "8 sequences")
