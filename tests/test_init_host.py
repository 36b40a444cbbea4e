"""The library's host weight generator (csrc/init_weights.cpp, built with the
library's own flags) equals the oracle's independent implementation of the init
spec bit for bit -- checked on the CPU, no GPU needed."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

from oracle import init_spec as I
from paper_2503_05130_amd import build as B

WRAP = r'''
#include "init_weights.h"
extern "C" {
void t_matrix(uint64_t seed, uint32_t layer, uint32_t slot, uint32_t in_dim, uint32_t out_dim,
              uint32_t qk_cols, float s, float sqk, uint16_t *dst) {
    iefwd::generate_matrix_transposed(iefwd::tensor_key(seed, layer, slot), in_dim, out_dim, qk_cols,
                                      (double)s, (double)sqk, dst);
}
void t_vec16(uint64_t seed, uint32_t layer, uint32_t slot, uint32_t n, float s, uint16_t *dst) {
    iefwd::generate_vector_bf16(iefwd::tensor_key(seed, layer, slot), n, (double)s, dst);
}
void t_vec32(uint64_t seed, uint32_t layer, uint32_t slot, uint32_t n, double off, float s, float *dst) {
    iefwd::generate_vector_f32(iefwd::tensor_key(seed, layer, slot), n, off, (double)s, dst);
}
uint64_t t_key(uint64_t seed, uint32_t layer, uint32_t slot) { return iefwd::tensor_key(seed, layer, slot); }
}
'''


@pytest.fixture(scope="module")
def libgen(tmp_path_factory):
    d = tmp_path_factory.mktemp("gen")
    wrap = d / "wrap.cpp"
    wrap.write_text(WRAP)
    so = d / "libgen.so"
    flags = [f for f in B.COMMON if not f.startswith("--offload-arch")] + B.PER_FILE["init_weights.cpp"]
    # host-only build of the same source with the library's flags
    cmd = [B.hipcc(), "--offload-arch=gfx950", "-shared"] + flags + ["-x", "hip",
           os.path.join(B.CSRC, "init_weights.cpp"), str(wrap), "-o", str(so)]
    subprocess.run(cmd, check=True, capture_output=True)
    lib = ctypes.CDLL(str(so))
    u64, u32, f32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.c_void_p
    lib.t_matrix.argtypes = [u64, u32, u32, u32, u32, u32, f32, f32, vp]
    lib.t_vec16.argtypes = [u64, u32, u32, u32, f32, vp]
    lib.t_vec32.argtypes = [u64, u32, u32, u32, ctypes.c_double, f32, vp]
    lib.t_key.restype = u64
    lib.t_key.argtypes = [u64, u32, u32]
    return lib


def test_keys(libgen, oracle_built):
    for seed in (0, 2, 53, 2 ** 64 - 3):
        for layer in (0, 11, 24):
            for slot in range(16):
                assert libgen.t_key(seed, layer, slot) == I.tensor_key(seed, layer, slot)


@pytest.mark.parametrize("seed,layer,slot,rows,cols,qk,s,sqk", [
    (2, 0, 0, 768, 2304, 1536, 0.02, 0.0),       # BERT-base QKV, default init
    (1, 0, 0, 128, 384, 256, 0.02, 0.06),        # stress init: Q/K blocks at 0.06
    (53, 23, 6, 256, 1024, 0, 0.02, 0.0),
    (4, 3, 8, 512, 128, 0, 0.3, 0.0),
    (7, 24, 14, 768, 2, 0, 0.02, 0.0),           # head
])
def test_matrices_bitwise(libgen, oracle_built, seed, layer, slot, rows, cols, qk, s, sqk):
    out = np.empty((cols, rows), np.uint16)      # library layout: output-major
    libgen.t_matrix(seed, layer, slot, rows, cols, qk, s, sqk, out.ctypes.data)
    s32, q32 = float(np.float32(s)), float(np.float32(sqk))
    ref = I.gen_weight_bits(seed, layer, slot, rows, cols, s32, qk_cols=qk, sigma_qk=q32)
    assert np.array_equal(out.T, ref)


@pytest.mark.parametrize("n,s", [(3072, 0.02), (2304, 0.0), (17, 0.5)])
def test_vectors_bitwise(libgen, oracle_built, n, s):
    out = np.empty(n, np.uint16)
    libgen.t_vec16(9, 1, 7, n, s, out.ctypes.data)
    assert np.array_equal(out, I.gen_weight_bits(9, 1, 7, 1, n, float(np.float32(s)))[0])
    g = np.empty(n, np.float32)
    libgen.t_vec32(9, 1, 4, n, 1.0, s, g.ctypes.data)
    assert np.array_equal(g.astype(np.float64), I.gen_ln_param(9, 1, 4, n, 1.0, float(np.float32(s))))
