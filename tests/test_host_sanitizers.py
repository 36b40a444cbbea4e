"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU needed): the host sources are compiled with hipcc, the
sanitizers on the host side only (each -fsanitize= after -Xarch_host), and
linked with the ordinarily built device objects and tests/c/sanitize_host.cpp,
which exercises the ABI's argument validation, the CU-mask builder, the quota
controller and the weight generator with exactly sized heap buffers."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2503_05130_amd", "csrc")
BUILD = os.path.join(ROOT, "paper_2503_05130_amd", "_build")
HOST_SOURCES = ["quota.cpp", "controller.cpp", "init_weights.cpp", "iefwd.cpp"]
DEVICE_OBJECTS = ["gemm.hip.o", "attention.hip.o", "decode.hip.o", "layernorm.hip.o", "train.hip.o"]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-Wall", "-Werror",
         "-Wno-unused-command-line-argument", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def hipcc():
    for cand in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not available")


def run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"
    return res


@pytest.fixture(scope="module")
def device_objects():
    objs = [os.path.join(BUILD, o) for o in DEVICE_OBJECTS]
    if not all(os.path.exists(o) for o in objs):
        from paper_2503_05130_amd import build as B
        B.build()
    return objs


def test_instrumentation_is_active(tmp_path):
    # a planted heap overflow, built with the same flags, must be reported
    src = tmp_path / "overflow.cpp"
    src.write_text("#include <cstdlib>\nint main(int c, char **) { int *p = (int *)std::malloc(4 * sizeof(int));"
                   " int v = p[c + 3]; std::free(p); return v == 12345; }\n")
    exe = tmp_path / "overflow"
    run([hipcc()] + FLAGS + SAN + ["-c", str(src), "-o", str(tmp_path / "overflow.o")])
    run([hipcc(), "--offload-arch=gfx950"] + SAN[:4] + [str(tmp_path / "overflow.o"), "-o", str(exe)])
    res = subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=60)
    assert res.returncode != 0 and "heap-buffer-overflow" in res.stderr


def test_host_code_clean_under_sanitizers(tmp_path, device_objects):
    objs = []
    for src in HOST_SOURCES:
        obj = str(tmp_path / (src + ".o"))
        extra = ["-ffp-contract=off"] if src == "init_weights.cpp" else []
        run([hipcc()] + FLAGS + SAN + extra + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    drv = str(tmp_path / "sanitize_host.o")
    run([hipcc()] + FLAGS + SAN + ["-c", os.path.join(ROOT, "tests", "c", "sanitize_host.cpp"), "-o", drv])
    exe = str(tmp_path / "sanitize_host")
    run([hipcc(), "--offload-arch=gfx950"] + SAN[:4] + [drv] + objs + device_objects + ["-o", exe])
    res = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=600)
    print(res.stdout, res.stderr)
    assert res.returncode == 0, res.stderr[-4000:]
    assert "host sanitizer checks passed" in res.stdout
