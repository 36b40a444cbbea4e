"""The plain-C ABI client builds and runs without Python in its process: with
a GPU it succeeds, without one it exits 3 with the library's ENODEV status on
stderr (a clean error, not a crash)."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CLIENT = os.path.join(HERE, "c", "abi_client")


def test_c_client_runs_or_reports_no_device(tmp_path):
    assert os.path.exists(CLIENT), "tests/c/abi_client is missing: run __graft_entry__.build()"
    res = subprocess.run([CLIENT, str(tmp_path / "logits.f32")], capture_output=True, text=True, timeout=120)
    if res.returncode == 0:
        assert os.path.getsize(tmp_path / "logits.f32") == 2 * 32 * 2 * 4
    else:
        assert res.returncode == 3 and "IEFWD_ENODEV" in res.stderr, (res.returncode, res.stderr)


def test_c_client_usage_error():
    res = subprocess.run([CLIENT], capture_output=True, text=True, timeout=60)
    assert res.returncode == 2 and "usage" in res.stderr
