"""Python binding of libiefwd (include/iefwd.h): argument marshalling only.

Every step of the forward pass runs in the library's HIP kernels; this module
converts Python arguments to C ones and turns non-zero status codes into
``IefwdError``.  torch supplies device memory and streams (``tensor.data_ptr()``,
``torch.cuda.Stream.cuda_stream``).

torch is imported before the library is loaded so that the library binds to the
HIP runtime torch already loaded (one runtime per process).  There is no CPU
fallback: if ``libiefwd.so`` is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # noqa: F401  (must be loaded before libiefwd.so)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libiefwd.so")

ABI_VERSION = 1
OK, EINVAL, ENODEV, ENOMEM, EHIP, ESTATE, EVERSION = 0, -1, -2, -3, -4, -5, -6
K_QKV, K_ATTN, K_OUTPROJ, K_FFN1, K_FFN2, K_LN, K_BWD_GEMM, K_BWD, K_OPTIM = range(9)
TRAIN_MASTER, TRAIN_GRAD, TRAIN_MOMENT1, TRAIN_MOMENT2 = range(4)
EPI_BIAS_BF16, EPI_BIAS_GELU_BF16, EPI_BIAS_RESID_F32 = 0, 1, 2

_u32, _u64, _i32, _f32, _vp, _sz = (ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int, ctypes.c_float,
                                    ctypes.c_void_p, ctypes.c_size_t)

# every function the header declares, with its C signature
SIGNATURES = {
    "iefwd_config_init": (None, [_vp]),
    "iefwd_device_info": (_i32, [_i32, ctypes.POINTER(_u32), ctypes.POINTER(_u32)]),
    "iefwd_build_cu_mask": (_i32, [_u32, _u32, _u32, _u32, ctypes.POINTER(_u32), _u32]),
    "iefwd_create": (_i32, [_vp, _i32, ctypes.POINTER(_vp)]),
    "iefwd_destroy": (_i32, [_vp]),
    "iefwd_set_quota": (_i32, [_vp, _u32]),
    "iefwd_set_quota_at": (_i32, [_vp, _u32, _u32]),
    "iefwd_decode": (_i32, [_vp, _vp, _u32, _u32, _i32]),
    "iefwd_prepare_quota_at": (_i32, [_vp, _u32, _u32]),
    "iefwd_set_stream_cache": (_i32, [_vp, _u32]),
    "iefwd_kernels_launched": (_i32, [_vp, ctypes.POINTER(ctypes.c_uint64)]),
    "iefwd_ctl_params_init": (_i32, [_vp]),
    "iefwd_ctl_create": (_i32, [_vp, ctypes.POINTER(_vp)]),
    "iefwd_ctl_destroy": (_i32, [_vp]),
    "iefwd_ctl_add": (_i32, [_vp, ctypes.c_double, ctypes.c_double, ctypes.c_int, ctypes.POINTER(_u32)]),
    "iefwd_ctl_report": (_i32, [_vp, _u32, ctypes.c_uint64, ctypes.c_double]),
    "iefwd_ctl_issue": (_i32, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_u32), ctypes.POINTER(_u32),
                                _u32]),
    "iefwd_ctl_state": (_i32, [_vp, ctypes.POINTER(ctypes.c_int32)]),
    "iefwd_set_cu_mask": (_i32, [_vp, ctypes.POINTER(_u32), _u32]),
    "iefwd_get_cu_mask": (_i32, [_vp, ctypes.POINTER(_u32), _u32]),
    "iefwd_submit": (_i32, [_vp, _vp, _u32, _u32, _i32]),
    "iefwd_wait": (_i32, [_vp]),
    "iefwd_read_logits": (_i32, [_vp, _vp, _sz, _i32]),
    "iefwd_last_batch_ms": (_i32, [_vp, ctypes.POINTER(_f32)]),
    "iefwd_get_stream": (_i32, [_vp, ctypes.POINTER(_vp)]),
    "iefwd_time_kernel": (_i32, [_vp, _u32, _i32]),
    "iefwd_kernel_time": (_i32, [_vp, _u32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_u64)]),
    "iefwd_export_tensor": (_i32, [_vp, _u32, _u32, _vp, _sz]),
    "iefwd_train_params_init": (None, [_vp]),
    "iefwd_train_create": (_i32, [_vp, _vp, _i32, ctypes.POINTER(_vp)]),
    "iefwd_train_step": (_i32, [_vp, _vp, _vp, _u32, _u32, _i32]),
    "iefwd_train_loss": (_i32, [_vp, ctypes.POINTER(_f32)]),
    "iefwd_train_steps": (_i32, [_vp, ctypes.POINTER(_u64)]),
    "iefwd_train_export": (_i32, [_vp, _u32, _u32, _u32, _vp, _sz]),
    "iefwd_last_error": (ctypes.c_char_p, []),
    "iefwd_status_string": (ctypes.c_char_p, [_i32]),
    "iefwd_test_gemm": (_i32, [_u32, _vp, _vp, _vp, _vp, _vp, _u32, _u32, _u32, _vp]),
    "iefwd_test_gemm_plan": (_i32, [_u32, _u32, _u32, _u32, _u32, _u32, ctypes.POINTER(_u32), ctypes.POINTER(_u32),
                                     ctypes.POINTER(_u32), ctypes.POINTER(_u32)]),
    "iefwd_test_gemm_skinny": (_i32, [_u32, _vp, _vp, _vp, _vp, _vp, _u32, _u32, _u32, _vp, _vp, _vp, _f32, _vp]),
    "iefwd_test_skinny_pack": (_i32, [_vp, _vp, _u32, _u32, _u32, _vp]),
    "iefwd_test_gemm_skinny_packed": (_i32, [_u32, _vp, _vp, _u32, _vp, _vp, _vp, _u32, _u32, _u32, _vp, _vp, _vp,
                                             _f32, _vp]),
    "iefwd_test_skinny_groups": (_i32, [_u32, _u32, _u32, _i32, ctypes.POINTER(_u32)]),
    "iefwd_test_gemm_qkv": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _u32, _u32, _u32, _u32, _vp]),
    "iefwd_test_attention": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _u32, _i32, _vp]),
    "iefwd_test_layernorm": (_i32, [_vp, _vp, _vp, _vp, _vp, _u32, _u32, _f32, _vp]),
    "iefwd_test_ln_head": (_i32, [_vp, _vp, _vp, _vp, _vp, _vp, _u32, _u32, _u32, _f32, _vp]),
    "iefwd_test_cu_probe": (_i32, [_vp, _u32, _vp]),
    "iefwd_test_decode_attention": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _u32, _u32, _u32, _vp]),
    "iefwd_decode_attention_noalloc": (_i32, [_vp, _vp, _vp, _vp, _u32, _u32, _u32, _u32, _u32, _u32, _vp]),
}


class Config(ctypes.Structure):
    """Mirror of ``iefwd_config``."""
    _fields_ = [
        ("abi_version", _u32), ("n_layers", _u32), ("d_model", _u32), ("n_heads", _u32),
        ("d_ff", _u32), ("max_batch", _u32), ("max_seq", _u32), ("n_out", _u32),
        ("pre_ln", _u32), ("causal", _u32), ("kv_cache", _u32),
        ("ln_eps", _f32), ("w_std", _f32), ("b_std", _f32), ("ln_std", _f32), ("qk_std", _f32),
        ("seed", _u64),
    ]


class IefwdError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func}: {status_string(status)} ({status}): {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2503_05130_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(status: int) -> str:
    return lib().iefwd_status_string(status).decode()


def last_error() -> str:
    return lib().iefwd_last_error().decode()


def _check(status: int, func: str) -> None:
    if status != OK:
        raise IefwdError(status, func, last_error())


def _ptr(x) -> int | None:
    """Device/host address of a tensor or array (None stays NULL)."""
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return int(x)


def _stream(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, torch.cuda.Stream):
        return s.cuda_stream
    return int(s)


# ------------------------------------------------------------------------------------ device
def device_info(device: int = 0) -> tuple[int, int]:
    n_cu, n_xcd = _u32(), _u32()
    _check(lib().iefwd_device_info(device, ctypes.byref(n_cu), ctypes.byref(n_xcd)), "iefwd_device_info")
    return n_cu.value, n_xcd.value


def build_cu_mask(n_cu: int, n_xcd: int, quota: int, first: int = 0, n_words: int | None = None) -> list[int]:
    n_words = n_words if n_words is not None else (n_cu + 31) // 32
    buf = (_u32 * n_words)()
    _check(lib().iefwd_build_cu_mask(n_cu, n_xcd, quota, first, buf, n_words), "iefwd_build_cu_mask")
    return list(buf)


def make_config(**kw) -> Config:
    cfg = Config()
    lib().iefwd_config_init(ctypes.byref(cfg))
    for k, v in kw.items():
        if not hasattr(cfg, k):
            raise KeyError(f"unknown config field {k}")
        setattr(cfg, k, v)
    return cfg


# ---------------------------------------------------------------------------------- instance
class Instance:
    """One serverless DL instance: its model, workspace and CU-masked stream."""

    def __init__(self, device: int = 0, **config):
        self._h = None
        self.cfg = make_config(**config)
        h = _vp()
        _check(lib().iefwd_create(ctypes.byref(self.cfg), device, ctypes.byref(h)), "iefwd_create")
        self._h = h
        self.device = device

    @property
    def out_width(self) -> int:
        return self.cfg.n_out if self.cfg.n_out > 0 else self.cfg.d_model

    def close(self) -> None:
        if self._h is not None:
            _check(lib().iefwd_destroy(self._h), "iefwd_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_quota(self, n_cu: int, first: int = 0) -> None:
        _check(lib().iefwd_set_quota_at(self._h, n_cu, first), "iefwd_set_quota_at")

    def prepare_quota(self, n_cu: int, first: int = 0) -> None:
        """Create the masked stream for (n_cu, first) ahead of time; may be called
        from another thread while this instance serves."""
        _check(lib().iefwd_prepare_quota_at(self._h, n_cu, first), "iefwd_prepare_quota_at")

    def set_stream_cache(self, capacity: int) -> None:
        """Number of masked streams (hardware queues) the instance keeps cached."""
        _check(lib().iefwd_set_stream_cache(self._h, capacity), "iefwd_set_stream_cache")

    def set_cu_mask(self, mask) -> None:
        buf = (_u32 * len(mask))(*mask)
        _check(lib().iefwd_set_cu_mask(self._h, buf, len(mask)), "iefwd_set_cu_mask")

    def get_cu_mask(self, n_words: int = 8) -> list[int]:
        buf = (_u32 * n_words)()
        _check(lib().iefwd_get_cu_mask(self._h, buf, n_words), "iefwd_get_cu_mask")
        return list(buf)

    def submit(self, x, batch: int | None = None, seq: int | None = None) -> None:
        """x: fp32 [batch, seq, d_model] -- a CUDA tensor (kept alive by the caller
        until wait/read) or a host array/tensor (copied before return)."""
        if isinstance(x, torch.Tensor):
            if x.dtype != torch.float32 or not x.is_contiguous():
                raise ValueError("x must be a contiguous float32 tensor")
            is_dev = 1 if x.is_cuda else 0
        else:
            x = np.ascontiguousarray(x, dtype=np.float32)
            is_dev = 0
        b = batch if batch is not None else x.shape[0]
        s = seq if seq is not None else x.shape[1]
        if int(np.prod(x.shape)) != b * s * self.cfg.d_model:
            raise ValueError("x does not have batch * seq * d_model elements")
        self._x_keep = x
        _check(lib().iefwd_submit(self._h, _ptr(x), b, s, is_dev), "iefwd_submit")
        self._last_shape = (b, s)

    def decode(self, x, pos: int) -> None:
        """One decode step (kv_cache instances): x fp32 [batch, d_model] -- the new
        tokens' embeddings -- appended at position `pos`."""
        if isinstance(x, torch.Tensor):
            if x.dtype != torch.float32 or not x.is_contiguous():
                raise ValueError("x must be a contiguous float32 tensor")
            is_dev = 1 if x.is_cuda else 0
        else:
            x = np.ascontiguousarray(x, dtype=np.float32)
            is_dev = 0
        b = x.shape[0]
        if int(np.prod(x.shape)) != b * self.cfg.d_model:
            raise ValueError("x does not have batch * d_model elements")
        self._x_keep = x
        _check(lib().iefwd_decode(self._h, _ptr(x), b, pos, is_dev), "iefwd_decode")
        self._last_shape = (b, 1)

    def wait(self) -> None:
        _check(lib().iefwd_wait(self._h), "iefwd_wait")

    def read_logits(self, out=None):
        """Waits and returns the last batch's output (numpy fp32 unless `out`
        -- a CUDA tensor or host array of the right size -- is given)."""
        b, s = getattr(self, "_last_shape", (0, 0))
        if out is None:
            out = np.empty((b, s, self.out_width), dtype=np.float32)
        is_dev = 1 if isinstance(out, torch.Tensor) and out.is_cuda else 0
        n = out.numel() if isinstance(out, torch.Tensor) else out.size
        _check(lib().iefwd_read_logits(self._h, _ptr(out), n, is_dev), "iefwd_read_logits")
        return out

    def last_batch_ms(self) -> float:
        v = _f32()
        _check(lib().iefwd_last_batch_ms(self._h, ctypes.byref(v)), "iefwd_last_batch_ms")
        return v.value

    def kernels_launched(self) -> int:
        v = _u64()
        _check(lib().iefwd_kernels_launched(self._h, ctypes.byref(v)), "iefwd_kernels_launched")
        return v.value

    def stream_handle(self) -> int:
        v = _vp()
        _check(lib().iefwd_get_stream(self._h, ctypes.byref(v)), "iefwd_get_stream")
        return v.value or 0

    def time_kernel(self, kind: int, enable: bool = True) -> None:
        _check(lib().iefwd_time_kernel(self._h, kind, 1 if enable else 0), "iefwd_time_kernel")

    def kernel_time(self, kind: int) -> tuple[float, int]:
        ms, n = ctypes.c_double(), _u64()
        _check(lib().iefwd_kernel_time(self._h, kind, ctypes.byref(ms), ctypes.byref(n)), "iefwd_kernel_time")
        return ms.value, n.value

    def export_tensor(self, layer: int, slot: int) -> np.ndarray:
        """Stored tensor in its logical layout: bf16 tensors as uint16 bit
        patterns, LN parameters as float32."""
        c = self.cfg
        d, F, n_out = c.d_model, c.d_ff, c.n_out
        shapes = {0: (d, 3 * d), 1: (3 * d,), 2: (d, d), 3: (d,), 4: (d,), 5: (d,), 6: (d, F), 7: (F,),
                  8: (F, d), 9: (d,), 10: (d,), 11: (d,), 12: (d,), 13: (d,), 14: (d, n_out), 15: (n_out,)}
        f32_slots = {4, 5, 10, 11, 12, 13}
        out = np.empty(shapes[slot], dtype=np.float32 if slot in f32_slots else np.uint16)
        _check(lib().iefwd_export_tensor(self._h, layer, slot, out.ctypes.data, out.nbytes),
               "iefwd_export_tensor")
        return out


# ---------------------------------------------------------------------- per-kernel entry points
def test_gemm(epilogue, a, w, bias, resid, out, M, N, K, stream=None) -> None:
    _check(lib().iefwd_test_gemm(epilogue, _ptr(a), _ptr(w), _ptr(bias), _ptr(resid), _ptr(out), M, N, K,
                                 _stream(stream)), "iefwd_test_gemm")


def test_gemm_skinny(epilogue, a, w, bias, resid, out, M, N, K, ln=None, stream=None) -> None:
    """ln: None, or (z, gamma, beta, eps) to take the activations as LayerNorm(z)."""
    z, g, b, eps = ln if ln is not None else (None, None, None, 0.0)
    _check(lib().iefwd_test_gemm_skinny(epilogue, _ptr(a), _ptr(w), _ptr(bias), _ptr(resid), _ptr(out), M, N, K,
                                        _ptr(z), _ptr(g), _ptr(b), eps, _stream(stream)), "iefwd_test_gemm_skinny")


def test_skinny_pack(w, dst, N, K, groups, stream=None) -> None:
    """dst (N * K bf16, device) = W [N, K] in the decode product's packed layout for `groups` K-groups."""
    _check(lib().iefwd_test_skinny_pack(_ptr(w), _ptr(dst), N, K, groups, _stream(stream)), "iefwd_test_skinny_pack")


def test_gemm_skinny_packed(epilogue, a, w_packed, groups, bias, resid, out, M, N, K, ln=None, stream=None) -> None:
    """test_gemm_skinny reading the packed copy of W (test_skinny_pack)."""
    z, g, b, eps = ln if ln is not None else (None, None, None, 0.0)
    _check(lib().iefwd_test_gemm_skinny_packed(epilogue, _ptr(a), _ptr(w_packed), groups, _ptr(bias), _ptr(resid),
                                               _ptr(out), M, N, K, _ptr(z), _ptr(g), _ptr(b), eps, _stream(stream)),
           "iefwd_test_gemm_skinny_packed")


def test_skinny_groups(M, N, K, ln) -> int:
    """The K-group count the decode product uses for (M, N, K), with or without the LayerNorm prologue."""
    g = _u32()
    _check(lib().iefwd_test_skinny_groups(M, N, K, 1 if ln else 0, ctypes.byref(g)), "iefwd_test_skinny_groups")
    return g.value


def test_gemm_qkv(a, w, bias, q, k, vt, batch, seq, d_model, n_heads, stream=None) -> None:
    _check(lib().iefwd_test_gemm_qkv(_ptr(a), _ptr(w), _ptr(bias), _ptr(q), _ptr(k), _ptr(vt), batch, seq,
                                     d_model, n_heads, _stream(stream)), "iefwd_test_gemm_qkv")


def test_attention(q, k, vt, ctx, batch, n_heads, seq, head_dim, causal, stream=None) -> None:
    _check(lib().iefwd_test_attention(_ptr(q), _ptr(k), _ptr(vt), _ptr(ctx), batch, n_heads, seq, head_dim,
                                      1 if causal else 0, _stream(stream)), "iefwd_test_attention")


def test_layernorm(z, gamma, beta, out_f32, out_bf16, rows, d, eps, stream=None) -> None:
    _check(lib().iefwd_test_layernorm(_ptr(z), _ptr(gamma), _ptr(beta), _ptr(out_f32), _ptr(out_bf16), rows,
                                      d, eps, _stream(stream)), "iefwd_test_layernorm")


def test_ln_head(z, gamma, beta, wh, bh, logits, rows, d, n_out, eps, stream=None) -> None:
    _check(lib().iefwd_test_ln_head(_ptr(z), _ptr(gamma), _ptr(beta), _ptr(wh), _ptr(bh), _ptr(logits), rows,
                                    d, n_out, eps, _stream(stream)), "iefwd_test_ln_head")


def test_decode_attention(q, k, vt, ctx, batch, n_heads, n_keys, head_dim, k_rows, vt_stride, stream=None) -> None:
    _check(lib().iefwd_test_decode_attention(_ptr(q), _ptr(k), _ptr(vt), _ptr(ctx), batch, n_heads, n_keys,
                                             head_dim, k_rows, vt_stride, _stream(stream)),
           "iefwd_test_decode_attention")


def test_gemm_plan(M: int, N: int, K: int, align: int, n_cu: int, ln_residual: bool = False) -> tuple[int, int, int, int]:
    """(k_order, tile_order, tile_m, tile_n) of an M x N x K product on n_cu CUs (ln_residual: the
    post-LN residual epilogue)."""
    o = [_u32() for _ in range(4)]
    _check(lib().iefwd_test_gemm_plan(M, N, K, align, n_cu, 1 if ln_residual else 0, *[ctypes.byref(v) for v in o]),
           "iefwd_test_gemm_plan")
    return tuple(v.value for v in o)


def decode_attention_noalloc(q, k, vt, ctx, batch, n_heads, n_keys, head_dim, k_rows, vt_stride,
                             stream=None) -> None:
    _check(lib().iefwd_decode_attention_noalloc(_ptr(q), _ptr(k), _ptr(vt), _ptr(ctx), batch, n_heads, n_keys,
                                                head_dim, k_rows, vt_stride, _stream(stream)),
           "iefwd_decode_attention_noalloc")


def test_cu_probe(n_groups: int, out, stream=None) -> None:
    _check(lib().iefwd_test_cu_probe(_stream(stream), n_groups, _ptr(out)), "iefwd_test_cu_probe")


# ------------------------------------------------------------------ quota controller
CTL_NONE, CTL_EMERGENCY, CTL_RECOVERY, CTL_CONTENTION = 0, 1, 2, 3


class TrainParams(ctypes.Structure):
    """Mirror of ``iefwd_train_params``."""
    _fields_ = [("abi_version", _u32), ("reserved0", _u32), ("lr", _f32), ("beta1", _f32), ("beta2", _f32),
                ("eps", _f32), ("weight_decay", _f32), ("reserved1", _f32)]


def train_params(**kw) -> TrainParams:
    tp = TrainParams()
    lib().iefwd_train_params_init(ctypes.byref(tp))
    for k, v in kw.items():
        if k not in ("lr", "beta1", "beta2", "eps", "weight_decay"):
            raise ValueError(f"unknown training parameter {k}")
        setattr(tp, k, v)
    return tp


class Trainer(Instance):
    """A training instance (post-LN encoder, softmax cross-entropy, AdamW): the
    same quota calls as an inference instance, plus whole training steps."""

    def __init__(self, device: int = 0, train: dict | None = None, **config):
        self._h = None
        self.cfg = make_config(**config)
        self.tp = train_params(**(train or {}))
        h = _vp()
        _check(lib().iefwd_train_create(ctypes.byref(self.cfg), ctypes.byref(self.tp), device, ctypes.byref(h)),
               "iefwd_train_create")
        self._h = h
        self.device = device

    def step(self, x, labels) -> None:
        """One asynchronous training step.  x fp32 [B, S, d], labels int32 [B, S]:
        both CUDA tensors (kept alive until the step completes) or both host arrays."""
        if isinstance(x, torch.Tensor) and x.is_cuda:
            if not (isinstance(labels, torch.Tensor) and labels.is_cuda):
                raise ValueError("x and labels must both be on the device or both on the host")
            if x.dtype != torch.float32 or not x.is_contiguous():
                raise ValueError("x must be a contiguous float32 tensor")
            if labels.dtype != torch.int32 or not labels.is_contiguous():
                raise ValueError("labels must be a contiguous int32 tensor")
            is_dev = 1
        else:
            x = np.ascontiguousarray(x.cpu().numpy() if isinstance(x, torch.Tensor) else x, dtype=np.float32)
            labels = np.ascontiguousarray(labels.cpu().numpy() if isinstance(labels, torch.Tensor) else labels,
                                          dtype=np.int32)
            is_dev = 0
        b, s_ = x.shape[0], x.shape[1]
        _check(lib().iefwd_train_step(self._h, _ptr(x), _ptr(labels), b, s_, is_dev), "iefwd_train_step")
        self._last_shape = (b, s_)
        self._keep = (x, labels)

    def loss(self) -> float:
        v = _f32()
        _check(lib().iefwd_train_loss(self._h, ctypes.byref(v)), "iefwd_train_loss")
        return float(v.value)

    def steps(self) -> int:
        v = _u64()
        _check(lib().iefwd_train_steps(self._h, ctypes.byref(v)), "iefwd_train_steps")
        return int(v.value)

    def export(self, layer: int, slot: int, what: int, shape) -> np.ndarray:
        out = np.empty(shape, dtype=np.float32)
        _check(lib().iefwd_train_export(self._h, layer, slot, what, out.ctypes.data, out.size), "iefwd_train_export")
        return out


CTL_TEMPORARY_YIELD = 1


class CtlParams(ctypes.Structure):
    _fields_ = [("abi_version", _u32), ("max_tokens", _u32), ("window", _u32), ("granule", _u32),
                ("min_quota", _u32), ("flags", _u32), ("eta_violation", ctypes.c_double),
                ("eta_increase", ctypes.c_double)]


class Controller:
    """The fast scale-up/down quota controller (iefwd_ctl_*): report each
    instance's kernels and last batch time once per control period, then
    issue() returns (tokens, quotas, first mask bits) in id order.
    temporary_yield=True sets IEFWD_CTL_TEMPORARY_YIELD."""

    def __init__(self, temporary_yield: bool = False, **params):
        p = CtlParams()
        _check(lib().iefwd_ctl_params_init(ctypes.byref(p)), "iefwd_ctl_params_init")
        for k, v in params.items():
            setattr(p, k, v)
        if temporary_yield:
            p.flags |= CTL_TEMPORARY_YIELD
        h = _vp()
        _check(lib().iefwd_ctl_create(ctypes.byref(p), ctypes.byref(h)), "iefwd_ctl_create")
        self._h = h.value
        self.n = 0

    def add(self, request: float, limit: float, slo_sensitive: bool) -> int:
        i = _u32()
        _check(lib().iefwd_ctl_add(self._h, request, limit, 1 if slo_sensitive else 0, ctypes.byref(i)),
               "iefwd_ctl_add")
        self.n += 1
        return i.value

    def report(self, i: int, kernels: int, klc_ms: float) -> None:
        _check(lib().iefwd_ctl_report(self._h, i, kernels, klc_ms), "iefwd_ctl_report")

    def issue(self) -> tuple[list[float], list[int], list[int]]:
        t, q, f = (ctypes.c_double * max(self.n, 1))(), (_u32 * max(self.n, 1))(), (_u32 * max(self.n, 1))()
        _check(lib().iefwd_ctl_issue(self._h, t, q, f, self.n), "iefwd_ctl_issue")
        return list(t)[:self.n], list(q)[:self.n], list(f)[:self.n]

    def state(self) -> int:
        v = ctypes.c_int32()
        _check(lib().iefwd_ctl_state(self._h, ctypes.byref(v)), "iefwd_ctl_state")
        return v.value

    def close(self) -> None:
        if getattr(self, "_h", None):
            lib().iefwd_ctl_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:   # interpreter shutdown
            pass

