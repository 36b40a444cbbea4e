"""Oracle side of the seeded random-init spec (test infrastructure only).

Two implementations of the same written definition:

* ``ref_*``  -- pure Python, one element at a time (``math.log``/``math.cos``
  are glibc's), rounding done by exact arithmetic rather than bit tricks.  Slow;
  used on small tensors to pin the fast path.
* ``gen_*``  -- the C routine in ``oracle/c/oracle_init.c`` through ctypes, for
  full-size models.

Definition (this project's reading; the paper fixes no initialisation, only
that each instance carries its own model weights, Sec. 3.2):

* mix64(z): SplitMix64 output function applied to z + 0x9E3779B97F4A7C15.
* tensor key = mix64(seed XOR mix64(32*layer + slot)); slots are listed in
  ``SLOTS``; model-global tensors use layer = n_layers.
* element e (row-major index in the logical [in, out] layout):
  a = mix64(key + 2e), b = mix64(key + 2e + 1),
  u1 = ((a >> 11) + 1) * 2^-53 in (0, 1], u2 = (b >> 11) * 2^-53,
  n = sqrt(-2 ln u1) * cos(2 pi u2)  (Box & Muller 1958), in fp64.
* weights/biases: sigma*n -> fp32 (RNE) -> bf16 (RNE).  LN gamma = 1 + ln_std*n,
  beta = ln_std*n, kept in fp32.
* the sigma values are the fp32 numbers a model config carries (its std fields
  are fp32), widened exactly to fp64: sigma = 0.02 means fl32(0.02).
"""
from __future__ import annotations

import ctypes
import math
import os
import struct
from fractions import Fraction

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15

SLOTS = dict(wqkv=0, bqkv=1, wo=2, bo=3, ln1_g=4, ln1_b=5, w1=6, b1=7, w2=8, b2=9,
             ln2_g=10, ln2_b=11, lnf_g=12, lnf_b=13, wh=14, bh=15)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_oracle_init.so")
_lib = None


# ----------------------------------------------------------------------------------
# pure-Python reference
# ----------------------------------------------------------------------------------
def ref_mix64(z: int) -> int:
    z = (z + GOLDEN) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def ref_tensor_key(seed: int, layer: int, slot: int) -> int:
    return ref_mix64((seed & MASK64) ^ ref_mix64(32 * layer + slot))


def ref_std_normal(key: int, e: int) -> float:
    a = ref_mix64((key + 2 * e) & MASK64)
    b = ref_mix64((key + 2 * e + 1) & MASK64)
    u1 = ((a >> 11) + 1) * 2.0 ** -53
    u2 = (b >> 11) * 2.0 ** -53
    return math.sqrt(-2.0 * math.log(u1)) * math.cos(6.283185307179586 * u2)


def ref_round_f32(x: float) -> float:
    """fp64 -> fp32, round to nearest even (C cast semantics)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def ref_round_bf16(f: float) -> float:
    """fp32 value -> nearest bf16 value, ties to even, by exact arithmetic.

    bf16 keeps 8 significant bits; the quantum at binary exponent e is
    2**(e-8) where f = m * 2**e, 0.5 <= |m| < 1.
    """
    if f == 0.0:
        return f
    m, e = math.frexp(f)
    q = Fraction(2) ** (e - 8)
    x = Fraction(f) / q                  # exact
    lo = math.floor(x)
    frac = x - lo
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    return float(lo * q)


def ref_weight(seed: int, layer: int, slot: int, rows: int, cols: int, sigma: float,
               qk_cols: int = 0, sigma_qk: float = 0.0) -> np.ndarray:
    key = ref_tensor_key(seed, layer, slot)
    out = np.empty(rows * cols, dtype=np.float64)
    for e in range(rows * cols):
        c = e % cols
        s = sigma_qk if (c < qk_cols and sigma_qk != 0.0) else sigma
        out[e] = ref_round_bf16(ref_round_f32(s * ref_std_normal(key, e)))
    return out.reshape(rows, cols)


def ref_ln_param(seed: int, layer: int, slot: int, n: int, offset: float, sigma: float) -> np.ndarray:
    key = ref_tensor_key(seed, layer, slot)
    return np.array([ref_round_f32(offset + sigma * ref_std_normal(key, e)) for e in range(n)])


# ----------------------------------------------------------------------------------
# fast path (C, glibc libm)
# ----------------------------------------------------------------------------------
def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build_c
            build_c.build()
        lib = ctypes.CDLL(_LIB_PATH)
        u64, u32, dbl = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_double
        lib.oracle_mix64.restype = u64
        lib.oracle_mix64.argtypes = [u64]
        lib.oracle_tensor_key.restype = u64
        lib.oracle_tensor_key.argtypes = [u64, u32, u32]
        lib.oracle_gen_bf16.restype = None
        lib.oracle_gen_bf16.argtypes = [u64, u64, u64, u64, dbl, dbl, ctypes.c_void_p]
        lib.oracle_gen_f32.restype = None
        lib.oracle_gen_f32.argtypes = [u64, u64, dbl, dbl, ctypes.c_void_p]
        lib.oracle_std_normals.restype = None
        lib.oracle_std_normals.argtypes = [u64, u64, ctypes.c_void_p]
        _lib = lib
    return _lib


def mix64(z: int) -> int:
    return int(_load().oracle_mix64(z & MASK64))


def tensor_key(seed: int, layer: int, slot: int) -> int:
    return int(_load().oracle_tensor_key(seed & MASK64, layer, slot))


def std_normals(key: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float64)
    _load().oracle_std_normals(key, n, out.ctypes.data)
    return out


def gen_weight_bits(seed: int, layer: int, slot: int, rows: int, cols: int, sigma: float,
                    qk_cols: int = 0, sigma_qk: float = 0.0) -> np.ndarray:
    """bf16 bit patterns (uint16) of a weight or bias, logical [rows, cols]."""
    out = np.empty((rows, cols), dtype=np.uint16)
    _load().oracle_gen_bf16(tensor_key(seed, layer, slot), rows, cols, qk_cols,
                            float(sigma), float(sigma_qk), out.ctypes.data)
    return out


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def gen_weight(seed, layer, slot, rows, cols, sigma, qk_cols=0, sigma_qk=0.0) -> np.ndarray:
    return bf16_bits_to_f64(gen_weight_bits(seed, layer, slot, rows, cols, sigma, qk_cols, sigma_qk))


def gen_ln_param(seed: int, layer: int, slot: int, n: int, offset: float, sigma: float) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    _load().oracle_gen_f32(tensor_key(seed, layer, slot), n, float(offset), float(sigma), out.ctypes.data)
    return out.astype(np.float64)


# ----------------------------------------------------------------------------------
# whole-model weights, one layer at a time (fp64 copies of the bf16/fp32 values)
# ----------------------------------------------------------------------------------
def _sigmas(shape: dict):
    """(w, b, ln, qk) standard deviations as the fp32 values of the config."""
    f32 = lambda v: float(np.float32(v))
    return (f32(shape["w_std"]), f32(shape["b_std"]), f32(shape["ln_std"]),
            f32(shape.get("qk_std", 0.0)))


def layer_weights(shape: dict, layer: int) -> dict:
    d, f, seed = shape["d_model"], shape["d_ff"], shape["seed"]
    ws, bs, ls, qk = _sigmas(shape)
    S = SLOTS
    return dict(
        wqkv=gen_weight(seed, layer, S["wqkv"], d, 3 * d, ws, qk_cols=2 * d, sigma_qk=qk),
        bqkv=gen_weight(seed, layer, S["bqkv"], 1, 3 * d, bs)[0],
        wo=gen_weight(seed, layer, S["wo"], d, d, ws),
        bo=gen_weight(seed, layer, S["bo"], 1, d, bs)[0],
        ln1_g=gen_ln_param(seed, layer, S["ln1_g"], d, 1.0, ls),
        ln1_b=gen_ln_param(seed, layer, S["ln1_b"], d, 0.0, ls),
        w1=gen_weight(seed, layer, S["w1"], d, f, ws),
        b1=gen_weight(seed, layer, S["b1"], 1, f, bs)[0],
        w2=gen_weight(seed, layer, S["w2"], f, d, ws),
        b2=gen_weight(seed, layer, S["b2"], 1, d, bs)[0],
        ln2_g=gen_ln_param(seed, layer, S["ln2_g"], d, 1.0, ls),
        ln2_b=gen_ln_param(seed, layer, S["ln2_b"], d, 0.0, ls),
    )


def global_weights(shape: dict) -> dict:
    d, L, seed = shape["d_model"], shape["n_layers"], shape["seed"]
    ws, bs, ls, _ = _sigmas(shape)
    out = dict(
        lnf_g=gen_ln_param(seed, L, SLOTS["lnf_g"], d, 1.0, ls),
        lnf_b=gen_ln_param(seed, L, SLOTS["lnf_b"], d, 0.0, ls),
    )
    n_out = shape["n_out"]
    if n_out > 0:
        out["wh"] = gen_weight(seed, L, SLOTS["wh"], d, n_out, ws)
        out["bh"] = gen_weight(seed, L, SLOTS["bh"], 1, n_out, bs)[0]
    return out


def ref_layer_weights(shape: dict, layer: int) -> dict:
    """Same tensors as ``layer_weights`` through the pure-Python path (tiny shapes only)."""
    d, f, seed = shape["d_model"], shape["d_ff"], shape["seed"]
    ws, bs, ls, qk = _sigmas(shape)
    S = SLOTS
    return dict(
        wqkv=ref_weight(seed, layer, S["wqkv"], d, 3 * d, ws, qk_cols=2 * d, sigma_qk=qk),
        bqkv=ref_weight(seed, layer, S["bqkv"], 1, 3 * d, bs)[0],
        wo=ref_weight(seed, layer, S["wo"], d, d, ws),
        bo=ref_weight(seed, layer, S["bo"], 1, d, bs)[0],
        ln1_g=ref_ln_param(seed, layer, S["ln1_g"], d, 1.0, ls),
        ln1_b=ref_ln_param(seed, layer, S["ln1_b"], d, 0.0, ls),
        w1=ref_weight(seed, layer, S["w1"], d, f, ws),
        b1=ref_weight(seed, layer, S["b1"], 1, f, bs)[0],
        w2=ref_weight(seed, layer, S["w2"], f, d, ws),
        b2=ref_weight(seed, layer, S["b2"], 1, d, bs)[0],
        ln2_g=ref_ln_param(seed, layer, S["ln2_g"], d, 1.0, ls),
        ln2_b=ref_ln_param(seed, layer, S["ln2_b"], d, 0.0, ls),
    )
