"""The ABI from plain C: tests/c/abi_client (built by __graft_entry__.build())
runs a two-layer encoder on a 64-CU quota from host memory in a process of its
own.  Its logits equal, bit for bit, what the Python binding gets for the same
config and input at the full quota, and match the fp64 oracle."""
import os
import subprocess

import numpy as np
import pytest

import paper_2503_05130_amd as ie
import workloads as W
from oracle import forward as F
from tests.gpu_util import instance_config, run_instance

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
CLIENT = os.path.join(HERE, "c", "abi_client")
B, S, D = 2, 32, 128


def client_input() -> np.ndarray:
    """x[i] = ((i * 7919) mod 2001 - 1000) / 1000 in fp32, as the C client computes it."""
    i = np.arange(B * S * D, dtype=np.int64)
    return (((i * 7919) % 2001 - 1000).astype(np.float32) / np.float32(1000)).reshape(B, S, D)


def test_c_client_matches_binding_and_oracle(tmp_path):
    assert os.path.exists(CLIENT), "tests/c/abi_client is missing: run __graft_entry__.build()"
    out_file = tmp_path / "logits.f32"
    print("running the C client", flush=True)
    res = subprocess.run([CLIENT, str(out_file)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    got = np.fromfile(out_file, dtype=np.float32).reshape(B, S, 2)
    shape = W.model_shape("encoder_l1_d128_s32_b2", n_layers=2, d_model=D, n_heads=2, d_ff=512, n_out=2,
                          pre_ln=0, causal=0, seed=7)
    x = client_input()
    with ie.Instance(**instance_config(shape, B, S)) as inst:
        mine = run_instance(inst, x)
    assert np.array_equal(got.view(np.uint32), mine.view(np.uint32))
    ref = F.forward(x, shape)
    assert F.max_abs(got, ref) <= 2e-2 and F.rel_l2(got, ref) <= 1e-2
