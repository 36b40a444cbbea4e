"""Host-side checks of the C ABI (no GPU needed): every declared symbol is
exported, the ctypes config mirror matches the C layout, the CU-mask builder,
and argument / state errors that are decided before any device work."""
import ctypes
import os
import re
import subprocess

import pytest
import torch

import paper_2503_05130_amd as ie

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "iefwd.h")
HAVE_GPU = torch.cuda.is_available()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(iefwd_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 20
    lib = ie.lib()
    for n in names:
        assert hasattr(lib, n), n
    # and the binding knows every one of them (and nothing else)
    assert sorted(ie.SIGNATURES) == names


def test_no_oracle_in_the_product():
    # the product library and binding never import, link or name the oracle
    for root, _, files in os.walk(os.path.join(ROOT, "paper_2503_05130_amd")):
        for f in files:
            path = os.path.join(root, f)
            if f.endswith(".py"):
                assert not re.search(r"^\s*(import|from)\s+oracle", open(path).read(), re.M), f
            elif f.endswith((".cpp", ".hip", ".h")):
                assert "oracle" not in open(path).read().lower(), f
    out = subprocess.run(["nm", "-D", ie.LIB_PATH], capture_output=True, text=True).stdout
    assert "oracle" not in out


def test_config_layout_matches_c(tmp_path):
    fields = [f for f, _ in ie.Config._fields_]
    prog = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "iefwd.h"', "int main(void) {",
             '  printf("size %zu\\n", sizeof(iefwd_config));']
    for f in fields:
        lines.append(f'  printf("{f} %zu\\n", offsetof(iefwd_config, {f}));')
    lines.append("  return 0; }")
    prog.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{ROOT}/include", str(prog), "-o", str(exe)],
                   check=True)
    out = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                       check=True).stdout.splitlines())
    assert int(out["size"]) == ctypes.sizeof(ie.Config)
    for f in fields:
        assert int(out[f]) == getattr(ie.Config, f).offset, f


def test_config_defaults():
    c = ie.make_config()
    assert c.abi_version == ie.ABI_VERSION
    assert c.ln_eps == pytest.approx(1e-5)
    assert c.w_std == pytest.approx(0.02)
    assert c.b_std == 0 and c.ln_std == 0 and c.qk_std == 0


def test_status_strings():
    assert ie.status_string(0) == "IEFWD_OK"
    assert ie.status_string(-1) == "IEFWD_EINVAL"
    assert ie.status_string(-6) == "IEFWD_EVERSION"
    assert ie.status_string(-99) == "IEFWD_UNKNOWN"


# ------------------------------------------------------------------------------ CU masks
def popcount(words):
    return sum(bin(w).count("1") for w in words)


def xcd_counts(words, n_cu, n_xcd):
    counts = [0] * n_xcd
    for b in range(n_cu):
        if (words[b // 32] >> (b % 32)) & 1:
            counts[b % n_xcd] += 1
    return counts


@pytest.mark.parametrize("q", [1, 7, 8, 64, 100, 128, 192, 255, 256])
def test_mask_balanced_over_xcds(q):
    m = ie.build_cu_mask(256, 8, q)
    assert len(m) == 8
    assert popcount(m) == q
    c = xcd_counts(m, 256, 8)
    assert max(c) - min(c) <= 1
    assert c == sorted(c, reverse=True)          # the extra CUs go to the first XCDs
    assert m == ie.build_cu_mask(256, 8, q)      # deterministic


def test_mask_nested_and_full():
    # a larger quota's mask contains every CU of a smaller one
    prev = [0] * 8
    for q in range(8, 257, 8):
        m = ie.build_cu_mask(256, 8, q)
        assert all((a & b) == a for a, b in zip(prev, m))
        prev = m
    assert ie.build_cu_mask(256, 8, 256) == [0xFFFFFFFF] * 8


def test_mask_extra_words_zeroed_and_errors():
    m = ie.build_cu_mask(256, 8, 16, n_words=10)
    assert m[8:] == [0, 0]
    for args in [(256, 8, 0), (256, 8, 257), (256, 0, 8), (250, 8, 8), (256, 8, 8, 256)]:
        with pytest.raises(ie.IefwdError) as e:
            ie.build_cu_mask(*args)
        assert e.value.status == ie.EINVAL
    with pytest.raises(ie.IefwdError):
        ie.build_cu_mask(256, 8, 8, n_words=7)


@pytest.mark.parametrize("q,first", [(64, 0), (64, 64), (100, 37), (192, 200), (256, 5), (1, 255), (24, 250)])
def test_mask_placed_balanced(q, first):
    # a run of q consecutive mask bits starting at `first` (cyclically) is
    # exactly bits first .. first + q - 1 mod 256, and within one CU per XCD
    m = ie.build_cu_mask(256, 8, q, first)
    bits = {b for b in range(256) if (m[b // 32] >> (b % 32)) & 1}
    assert bits == {(first + i) % 256 for i in range(q)}
    c = xcd_counts(m, 256, 8)
    assert max(c) - min(c) <= 1


def test_mask_packed_placements_disjoint():
    # instances packed one after another get disjoint CUs up to 256 CUs in
    # total and cover the device exactly when the quotas sum to 256
    for quotas in [(64, 192), (128, 128), (192, 64), (24, 40, 64, 128), (8,) * 32]:
        first, seen = 0, [0] * 8
        for q in quotas:
            m = ie.build_cu_mask(256, 8, q, first)
            assert all((a & b) == 0 for a, b in zip(seen, m))
            seen = [a | b for a, b in zip(seen, m)]
            first = (first + q) % 256
        assert seen == [0xFFFFFFFF] * 8


# ------------------------------------------------------------------------------ create errors
BASE = dict(n_layers=1, d_model=128, n_heads=2, d_ff=512, max_batch=2, max_seq=32)


@pytest.mark.parametrize("bad,status", [
    (dict(abi_version=2), ie.EVERSION),
    (dict(d_model=100), ie.EINVAL),
    (dict(n_heads=3), ie.EINVAL),
    (dict(n_heads=4), ie.EINVAL),          # head dim 32 unsupported
    (dict(d_ff=100), ie.EINVAL),
    (dict(n_out=17), ie.EINVAL),
    (dict(pre_ln=2), ie.EINVAL),
    (dict(max_batch=0), ie.EINVAL),
    (dict(n_layers=0), ie.EINVAL),
    (dict(ln_eps=0.0), ie.EINVAL),
    (dict(w_std=-1.0), ie.EINVAL),
    (dict(kv_cache=2), ie.EINVAL),
    (dict(kv_cache=1, pre_ln=0), ie.EINVAL),          # decode needs a causal pre-LN stack
    (dict(kv_cache=1, pre_ln=1, causal=0), ie.EINVAL),
    (dict(max_batch=1 << 16, max_seq=1 << 14), ie.EINVAL),
])
def test_create_rejects_bad_config(bad, status):
    cfg = dict(BASE, **bad)
    with pytest.raises(ie.IefwdError) as e:
        ie.Instance(**cfg)
    assert e.value.status == status
    assert ie.last_error() != ""


@pytest.mark.skipif(HAVE_GPU, reason="checks the no-device path")
def test_no_device_paths():
    with pytest.raises(ie.IefwdError) as e:
        ie.device_info(0)
    assert e.value.status == ie.ENODEV
    with pytest.raises(ie.IefwdError) as e:
        ie.Instance(**BASE)
    assert e.value.status == ie.ENODEV


def test_null_arguments():
    L = ie.lib()
    assert L.iefwd_create(None, 0, None) == ie.EINVAL
    assert L.iefwd_destroy(None) == ie.OK
    assert L.iefwd_set_quota(None, 8) == ie.EINVAL
    assert L.iefwd_set_quota_at(None, 8, 0) == ie.EINVAL
    assert L.iefwd_decode(None, None, 1, 0, 1) == ie.EINVAL
    assert L.iefwd_prepare_quota_at(None, 8, 0) == ie.EINVAL
    assert L.iefwd_set_stream_cache(None, 2) == ie.EINVAL
    assert L.iefwd_submit(None, None, 1, 1, 0) == ie.EINVAL
    assert L.iefwd_wait(None) == ie.EINVAL
    assert L.iefwd_read_logits(None, None, 0, 0) == ie.EINVAL
    assert L.iefwd_device_info(0, None, None) == ie.EINVAL
    assert "NULL" in ie.last_error()


def test_kernel_entry_points_validate_shapes():
    L = ie.lib()
    p = 0x1000  # never dereferenced: every call below fails validation first
    assert L.iefwd_test_gemm(9, p, p, p, p, p, 4, 64, 64, None) == ie.EINVAL      # epilogue
    assert L.iefwd_test_gemm(0, p, p, p, None, p, 4, 60, 64, None) == ie.EINVAL   # N % 64
    assert L.iefwd_test_gemm(0, p, p, p, None, p, 4, 64, 65, None) == ie.EINVAL   # K % 64
    assert L.iefwd_test_gemm(2, p, p, p, None, p, 4, 64, 64, None) == ie.EINVAL   # resid missing
    assert L.iefwd_test_attention(p, p, p, p, 1, 1, 8, 32, 0, None) == ie.EINVAL  # head dim
    assert L.iefwd_test_attention(p, p, p, p, 0, 1, 8, 64, 0, None) == ie.EINVAL  # empty
    assert L.iefwd_test_decode_attention(p, p, p, p, 1, 1, 8, 32, 8, 64, None) == ie.EINVAL    # head dim
    assert L.iefwd_test_decode_attention(p, p, p, p, 1, 1, 9000, 64, 9000, 9024, None) == ie.EINVAL  # > 8192 keys
    assert L.iefwd_test_decode_attention(p, p, p, p, 1, 1, 65, 64, 64, 128, None) == ie.EINVAL  # k_rows < keys
    assert L.iefwd_test_decode_attention(p, p, p, p, 1, 1, 8, 64, 8, 100, None) == ie.EINVAL   # stride % 64
    assert L.iefwd_test_layernorm(p, p, p, p, None, 4, 100, 1e-5, None) == ie.EINVAL
    assert L.iefwd_test_ln_head(p, p, p, p, p, p, 4, 128, 0, 1e-5, None) == ie.EINVAL
    assert L.iefwd_test_cu_probe(None, 0, p) == ie.EINVAL
    assert L.iefwd_test_gemm_qkv(p, p, p, p, p, p, 1, 4, 100, 2, None) == ie.EINVAL


# ------------------------------------------------------------------ training ABI (host-side decisions)
def test_train_params_layout_and_defaults(tmp_path):
    fields = [f for f, _ in ie.TrainParams._fields_]
    prog = tmp_path / "tlayout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "iefwd.h"', "int main(void) {",
             '  printf("size %zu\\n", sizeof(iefwd_train_params));']
    for f in fields:
        lines.append(f'  printf("{f} %zu\\n", offsetof(iefwd_train_params, {f}));')
    lines.append("  return 0; }")
    prog.write_text("\n".join(lines))
    exe = tmp_path / "tlayout"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{ROOT}/include", str(prog), "-o", str(exe)],
                   check=True)
    out = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                       check=True).stdout.splitlines())
    assert int(out["size"]) == ctypes.sizeof(ie.TrainParams)
    for f in fields:
        assert int(out[f]) == getattr(ie.TrainParams, f).offset, f
    tp = ie.train_params()
    assert tp.abi_version == ie.ABI_VERSION
    assert (tp.lr, tp.beta1, tp.beta2, tp.eps, tp.weight_decay) == pytest.approx((1e-4, 0.9, 0.999, 1e-8, 0.01))
    with pytest.raises(ValueError):
        ie.train_params(momentum=0.9)


TRAIN_BASE = dict(BASE, pre_ln=0, causal=0, n_out=2)


@pytest.mark.parametrize("bad", [
    dict(pre_ln=1),                         # post-LN stacks only
    dict(n_out=0),                          # needs a head (classes)
    dict(d_model=256, n_heads=2),           # head dim 128
    dict(max_seq=256),                      # attention backward covers S <= 128
])
def test_train_create_rejects_bad_config(bad):
    with pytest.raises(ie.IefwdError) as e:
        ie.Trainer(**dict(TRAIN_BASE, **bad))
    assert e.value.status == ie.EINVAL


@pytest.mark.parametrize("bad", [dict(lr=-1.0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=0.0),
                                 dict(weight_decay=float("nan"))])
def test_train_create_rejects_bad_params(bad):
    with pytest.raises(ie.IefwdError) as e:
        ie.Trainer(train=bad, **TRAIN_BASE)
    assert e.value.status == ie.EINVAL


def test_train_null_and_version():
    L = ie.lib()
    cfg = ie.make_config(**TRAIN_BASE)
    h = ctypes.c_void_p()
    assert L.iefwd_train_create(ctypes.byref(cfg), None, 0, ctypes.byref(h)) == ie.EINVAL
    assert h.value is None
    tp = ie.train_params()
    tp.abi_version = 99
    assert L.iefwd_train_create(ctypes.byref(cfg), ctypes.byref(tp), 0, ctypes.byref(h)) == ie.EVERSION
    assert L.iefwd_train_step(None, None, None, 1, 64, 0) == ie.EINVAL
    assert L.iefwd_train_loss(None, None) == ie.EINVAL
    assert L.iefwd_train_steps(None, None) == ie.EINVAL
    assert L.iefwd_train_export(None, 0, 0, 0, None, 0) == ie.EINVAL
