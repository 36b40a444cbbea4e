"""The documented limits, reached: the widest model (d_model 4096, head
dimension 128, the LayerNorm and skinny-prologue row limit), a long prefill
(4096 tokens, 64-key chunks), and decode steps on the widest model -- each
against the fp64 oracle."""
import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from tests.gpu_util import DEV, instance_config, run_instance
from tests.test_gpu_kernels import test_attention as _attention_case

pytestmark = pytest.mark.gpu

MAX_ABS, REL_L2 = 2e-2, 1e-2


def check(got, ref, what):
    ma, rl = F.max_abs(got, ref), F.rel_l2(got, ref)
    print(f"  {what}: max_abs={ma:.3e} rel_l2={rl:.3e}", flush=True)
    assert np.all(np.isfinite(got))
    assert ma <= MAX_ABS and rl <= REL_L2, (what, ma, rl)


def wide_shape(**over):
    return W.model_shape("encoder_l1_d128_s32_b2", **dict(dict(n_layers=1, d_model=4096, n_heads=32, d_ff=4096,
                                                               pre_ln=1, causal=1, n_out=4), **over))


def test_widest_model_forward():
    shape = wide_shape(pre_ln=0, causal=0)
    print("forward d_model 4096, post-LN", flush=True)
    x = W.make_input(411, 2, 24, 4096)
    with ie.Instance(**instance_config(shape, 2, 24)) as inst:
        check(run_instance(inst, x), F.forward(x, shape), "d4096 post-LN")


def test_widest_model_decode():
    """Prefill then decode steps on the d_model 4096 pre-LN decoder: the skinny
    products' LayerNorm prologue at its row limit (K = 4096, M * K = 16384 at 4
    sequences)."""
    shape = wide_shape()
    B, P, G = 4, 8, 2
    print("decode d_model 4096, 4 sequences", flush=True)
    x = W.make_input(412, B, P + G, 4096)
    with ie.Instance(**instance_config(shape, B, P + G), kv_cache=1) as inst:
        inst.submit(torch.from_numpy(np.ascontiguousarray(x[:, :P])).to(DEV))
        check(inst.read_logits(), F.forward(x[:, :P], shape), "prompt")
        for g in range(G):
            inst.decode(torch.from_numpy(np.ascontiguousarray(x[:, P + g])).to(DEV), P + g)
            check(inst.read_logits()[:, 0], F.forward(x[:, :P + g + 1], shape)[:, P + g], f"step {g}")


@pytest.mark.parametrize("causal", [False, True])
def test_long_prefill_attention(causal):
    """4096 keys per query: 64 chunks of the online softmax."""
    print(f"attention S=4096 causal={causal}", flush=True)
    _attention_case(1, 1, 4096, 128, causal, 1.0)
