"""HGSS inference profiling (Sec. 3.2): the search on synthetic latency
surfaces, pinned to the example path the paper prints, against a traversal."""
import math

import pytest

from paper_2503_05130_amd import profiler as P
from tests.golden_data import rows


def test_smr_to_cus():
    assert [P.smr_to_cus(s) for s in (10, 20, 30, 40, 50, 100)] == [24, 48, 80, 104, 128, 256]
    assert all(P.smr_to_cus(s) % 8 == 0 for s in range(1, 101))
    assert P.smr_to_cus(0.1) == 8


def test_paper_example_path():
    # the GPT2-large example of the draft text of Sec. 3.2 (100 ms SLO, tests/golden/hgss_printed_path.txt):
    # <1,10>, <2,20>, <4,30> meet the SLO, <8,40> violates it and the search stops there
    printed = [(int(b), float(s), m == "1") for b, s, m in rows("hgss_printed_path.txt")]

    def measure(ibs, smr):
        return 60.0 if ibs >= 8 else 20.0 * ibs / (smr / 10.0)
    r = P.hgss(measure, slo_ms=100.0)
    assert r["path"] == [(b, s) for b, s, _ in printed]
    assert [measure(b, s) <= 100.0 / 2 for b, s in r["path"]] == [m for _, _, m in printed]   # t_exec = SLO / 2
    assert r["trials"] == len(printed)
    # TE = IBS / (t * SMR): 1/(0.02*10) = 5, 2/(0.02*20) = 5, 4/(0.02667*30) = 5  -> ties: first max
    tes = [P.throughput_efficacy(b, measure(b, s), s) for b, s in r["path"][:3]]
    assert tes == pytest.approx([5.0, 5.0, 5.0])
    assert r["request_smr"] == 10.0 and r["limit_smr"] == 20.0


def test_request_is_max_te_and_limit_doubles():
    # batching helps sublinearly, SMR with diminishing returns
    def measure(ibs, smr):
        return 2.0 + 3.0 * ibs ** 0.6 * (100.0 / smr) ** 0.5
    r = P.hgss(measure, slo_ms=100.0, max_ibs=256)
    feas = [(b, s) for b, s in r["path"] if measure(b, s) <= 50.0]
    best = max(feas, key=lambda c: c[0] / (measure(*c) * 1e-3 * c[1]))
    assert (r["ibs"], r["request_smr"]) == best
    assert r["limit_smr"] == min(100.0, 2 * best[1])


def test_heavy_model_climbs_smr_first():
    # nothing fits at 10% for one sequence: SMR rises at IBS 1 until it does
    def measure(ibs, smr):
        return 800.0 * ibs / smr
    r = P.hgss(measure, slo_ms=100.0)
    assert r["path"][:3] == [(1, 10.0), (1, 20.0), (2, 30.0)]
    assert measure(*r["path"][0]) > 50.0 and measure(*r["path"][1]) <= 50.0


def test_never_feasible_ends_at_full_device():
    r = P.hgss(lambda b, s: 1e6, slo_ms=100.0)
    assert r["path"][-1] == (1, 100.0) and r.get("best") is None and r["trials"] == 10


def convex(ibs, smr):
    # batch time grows with IBS, falls with SM rate with diminishing returns
    return 1.5 + 0.25 * ibs * (100.0 / smr) ** 0.35 + 0.02 * ibs ** 1.3


def test_walks_against_traversal():
    ibs_list = [1 << k for k in range(9)]
    smr_list = [10.0 * k for k in range(1, 11)]
    t = P.traversal(convex, 100.0, ibs_list, smr_list)
    d = P.hgss(convex, 100.0, max_ibs=256)
    f = P.hgss(convex, 100.0, max_ibs=256, walk="frontier")
    assert t["trials"] == 90
    assert d["trials"] <= 10 and f["trials"] <= len(ibs_list) + len(smr_list)
    # the frontier walk reaches the traversal's optimum (it lies on the
    # smallest-feasible-SMR frontier); the printed diagonal cannot reach it
    assert f["best"]["te"] == pytest.approx(t["best"]["te"])
    assert (f["ibs"], f["request_smr"]) == (t["ibs"], t["request_smr"])
    assert d["best"]["te"] < t["best"]["te"]



def test_printed_traversal_grid_and_trial_counts():
    # Table "Inference function profiling comparison" (tests/golden/profiling_trials_table.txt):
    # the traversal costs 60 trials per model, HGSS 6 to 9.  The grid that gives 60 is IBS
    # 1 .. 32 (doubling) times SMR 10 .. 100 (steps of 10); on it the diagonal walk stays
    # within the printed HGSS counts for surfaces from light to heavy.
    table = {r[0]: [int(v) for v in r[1:]] for r in rows("profiling_trials_table.txt")}
    ibs_list = [1 << k for k in range(6)]
    smr_list = [10.0 * k for k in range(1, 11)]
    for scale in (0.5, 1.0, 4.0, 16.0):
        def m(b, s, sc=scale):
            return sc * convex(b, s)
        t = P.traversal(m, 100.0, ibs_list, smr_list)
        d = P.hgss(m, 100.0, max_ibs=32)
        assert t["trials"] == table["traversal"][0] == 60
        assert d["trials"] <= max(table["hgss"]), (scale, d["trials"])

def test_frontier_visits_smallest_feasible_smr_per_ibs():
    f = P.hgss(convex, 100.0, max_ibs=256, walk="frontier")
    seen = {}
    for b, s in f["path"]:
        if convex(b, s) <= 50.0:
            seen.setdefault(b, s)
    for b, s in seen.items():
        assert s == 10.0 or convex(b, s - 10.0) > 50.0


def test_unknown_walk_rejected():
    with pytest.raises(ValueError):
        P.hgss(convex, 100.0, walk="spiral")


# ------------------------------------------------------------------ training profiling (binary search)
def saturating(knee_cus, t_max=1000.0):
    """Throughput linear in the quota up to the knee, flat after it."""
    return lambda q: t_max * min(q, knee_cus) / knee_cus


def test_train_binary_search_follows_the_printed_rule():
    from paper_2503_05130_amd.profiler import train_binary_search
    calls = []

    def measure(q):
        calls.append(q)
        return saturating(128)(q)
    r = train_binary_search(measure, 0.8)
    # T1 at 100%, then mid = 50% (128 CUs): 1000 >= 800 + 20 -> high = 50; mid = 25% (64 CUs): 500 -> low = 25 ...
    assert calls[0] == 256 and calls[1] == 128 and calls[2] == 64
    assert abs(r["quota_cus"] - 0.8 * 128) <= 8             # the knee times p, to one XCD granule
    assert r["t1"] == 1000.0
    assert r["trials"] <= 8


def test_train_binary_search_stops_inside_the_band():
    from paper_2503_05130_amd.profiler import train_binary_search
    # saturating at 64 CUs: 50% is already full throughput, inside the p = 100% band: the printed rule stops there
    r = train_binary_search(saturating(64), 1.0)
    assert r["path"] == [(100.0, 256), (50.0, 128)] and r["quota_cus"] == 128
    # a knee above 50%: bisects upward until a setting is inside the band
    r = train_binary_search(saturating(200), 1.0)
    assert saturating(200)(r["quota_cus"]) >= 980.0 and r["quota_cus"] >= 200


def test_train_binary_search_tight_finds_the_knee():
    from paper_2503_05130_amd.profiler import train_binary_search
    for knee in (64, 96, 200, 256):
        r = train_binary_search(saturating(knee), 1.0, tight=True)
        assert knee - 16 <= r["quota_cus"] <= knee + 8, (knee, r)


def test_train_binary_search_against_traversal():
    import numpy as np

    from paper_2503_05130_amd.profiler import train_binary_search, train_traversal
    rng = np.random.default_rng(1)
    for _ in range(20):
        knee = int(rng.integers(2, 33)) * 8
        f = saturating(knee)
        for p in (0.8, 1.0):
            tv = train_traversal(f, p)
            assert tv["trials"] == 32
            for tight in (False, True):
                bs = train_binary_search(f, p, tight=tight)
                assert bs["trials"] < tv["trials"]
                # the setting delivers throughput no lower than the band below p * T1 (to one XCD granule)
                assert f(bs["quota_cus"]) >= (p - 0.02) * 1000.0 - 1000.0 * 8 / knee
                assert bs["quota_cus"] >= tv["quota_cus"] - 8
            assert abs(train_binary_search(f, p, tight=True)["quota_cus"] - tv["quota_cus"]) <= 16
