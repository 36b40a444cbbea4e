"""HGSS on a real instance (small model): every trial is a measured batch on
the requested CU quota; the chosen setting meets the SLO."""
import pytest

from paper_2503_05130_amd import profiler as P

pytestmark = pytest.mark.gpu


def test_hgss_on_small_encoder():
    shape = dict(n_layers=2, d_model=256, n_heads=4, d_ff=1024, pre_ln=0, causal=0, n_out=2)
    timer = P.InstanceTimer(shape, seq=64, max_ibs=64, seed=7, n_warm=1, n_time=3)
    try:
        r = P.hgss(timer, slo_ms=2.0, max_ibs=64)
        print(r, flush=True)
        assert r["trials"] >= 2
        assert r["best"] is not None and r["best"]["t_ms"] <= 1.0
        assert r["limit_smr"] == min(100.0, 2 * r["request_smr"])
        assert all(k in timer.cache for k in [tuple(p) for p in r["path"]])
    finally:
        timer.close()
