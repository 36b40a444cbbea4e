"""Seeded synthetic workloads shared by the tests, the bench and the oracle checks.

This module holds *only* shapes, seeds and the input generator. It contains none
of the forward-pass arithmetic, so both the HIP path and the CPU oracle can use
it without sharing any of the method's code.

Shapes follow the serving workloads of the paper's evaluation (Sec. 5.1,
"Workloads": BERT-base and RoBERTa-large class encoders, GPT2-large / LLaMA-class
decoders).  Trained weights and production traces are not available, so
weights come from the seeded random-init spec and inputs are i.i.d. N(0,1)
fp32 embeddings (no vocabulary, no positions, no padding).
"""
from __future__ import annotations

import numpy as np

# Each workload: model shape + the batch/seq it is run at + the weight seed.
# Keys of the model shape match the fields of the library's config struct.
WORKLOADS = {
    # single post-LN encoder layer, d=128, 2 heads (dh=64), FFN 512; returns hidden states
    "encoder_l1_d128_s32_b2": dict(
        n_layers=1, d_model=128, n_heads=2, d_ff=512, pre_ln=0, causal=0, n_out=0,
        seq=32, batch=2, seed=1, input_seed=1001),
    # BERT-base-shaped post-LN encoder stack, per-token 768->2 head
    "bert_base_l12_d768_s128": dict(
        n_layers=12, d_model=768, n_heads=12, d_ff=3072, pre_ln=0, causal=0, n_out=2,
        seq=128, batch=32, batches=(1, 8, 32), seed=2, input_seed=2000),
    # RoBERTa-large-sized causal pre-LN stack (prefill)
    "decoder_l24_d1024_s512": dict(
        n_layers=24, d_model=1024, n_heads=16, d_ff=4096, pre_ln=1, causal=1, n_out=2,
        seq=512, batch=8, seed=4, input_seed=4000),
    # large causal pre-LN stack, dh=128 (prefill)
    "decoder_l24_d2048_s1024": dict(
        n_layers=24, d_model=2048, n_heads=16, d_ff=8192, pre_ln=1, causal=1, n_out=2,
        seq=1024, batch=2, seed=53, input_seed=5300),
}

MODEL_KEYS = ("n_layers", "d_model", "n_heads", "d_ff", "pre_ln", "causal", "n_out")

# Stress init: non-zero biases, LN affine and sharper attention, so that a
# mistake in a bias add, an affine step, the score scale or the mask cannot
# hide behind near-uniform attention (zero biases, gamma=1, beta=0, std 0.02).
STRESS_INIT = dict(b_std=0.02, ln_std=0.02, qk_std=0.06)


def model_shape(name: str, **overrides) -> dict:
    """The model-shape part of a workload (plus init parameters), as a dict."""
    w = WORKLOADS[name]
    shape = {k: w[k] for k in MODEL_KEYS}
    shape.update(dict(ln_eps=1e-5, w_std=0.02, b_std=0.0, ln_std=0.0, qk_std=0.0, seed=w["seed"]))
    shape.update(overrides)
    return shape


def make_input(seed: int, batch: int, seq: int, d_model: int) -> np.ndarray:
    """fp32 [batch, seq, d_model] i.i.d. standard normal embeddings."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((batch, seq, d_model), dtype=np.float32)


def tiny_shape(pre_ln: int, causal: int, n_out: int = 0, seed: int = 7, **kw) -> dict:
    """A shape small enough for the pure-Python oracle (B=2, S=4, d=8, H=2, F=16)."""
    shape = dict(n_layers=2, d_model=8, n_heads=2, d_ff=16, pre_ln=pre_ln, causal=causal,
                 n_out=n_out, ln_eps=1e-5, w_std=0.3, b_std=0.1, ln_std=0.1, qk_std=0.0,
                 seed=seed)
    shape.update(kw)
    return shape


def make_labels(seed: int, batch: int, seq: int, n_classes: int) -> np.ndarray:
    """int32 [batch, seq] uniform class labels in [0, n_classes)."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_classes, size=(batch, seq), dtype=np.int32)
