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


def test_training_binary_search_on_small_encoder():
    """Binary search over CU quotas with real training steps: the request
    setting delivers (close to) 80% of the full-GPU throughput, the limit
    (close to) all of it, with fewer trials than a traversal."""
    shape = dict(n_layers=2, d_model=256, n_heads=4, d_ff=1024, pre_ln=0, causal=0, n_out=2)
    timer = P.TrainTimer(shape, seq=64, batch=8, seed=9)
    try:
        for p in (0.8, 1.0):
            r = P.train_binary_search(timer, p)
            print(p, r, flush=True)
            t = timer(r["quota_cus"])
            assert r["trials"] <= 8
            # a measured setting: inside the band, or the upper end of an adjacent pair
            assert t >= (p - 0.02) * r["t1"] * 0.9
            assert all(q in timer.cache for _, q in r["path"])
    finally:
        timer.close()
