"""Helpers shared by the GPU tests: bf16 staging through torch and the
instance-config conversion.  No forward-pass arithmetic lives here."""
from __future__ import annotations

import numpy as np
import torch

import paper_2503_05130_amd as ie

DEV = "cuda:0"


def bf16_round(x: np.ndarray) -> torch.Tensor:
    """fp32/fp64 array -> bf16 CPU tensor (round to nearest even)."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def to_dev(t: torch.Tensor) -> torch.Tensor:
    return t.contiguous().to(DEV)


def sync():
    torch.cuda.synchronize()


def instance_config(shape: dict, max_batch: int, max_seq: int) -> dict:
    keys = ("n_layers", "d_model", "n_heads", "d_ff", "pre_ln", "causal", "n_out", "ln_eps",
            "w_std", "b_std", "ln_std", "qk_std", "seed")
    cfg = {k: shape[k] for k in keys}
    cfg.update(max_batch=max_batch, max_seq=max_seq)
    return cfg


def run_instance(inst: "ie.Instance", x: np.ndarray) -> np.ndarray:
    """Submit one batch from device memory and read the output back."""
    xd = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV)
    inst.submit(xd)
    out = inst.read_logits()
    del xd
    return out


def compare(got: np.ndarray, ref: np.ndarray) -> tuple[float, float]:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = got - ref
    return float(np.max(np.abs(err))), float(np.linalg.norm(err) / np.linalg.norm(ref))
