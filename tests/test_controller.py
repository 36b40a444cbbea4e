"""Quota controller (Sec. 3.4.1, Alg. 2): the oracle pinned to the behaviour
the paper's text describes, and the library's controller (iefwd_ctl_*)
compared with the oracle on seeded random observation streams.  Host only."""
import math

import numpy as np
import pytest

import paper_2503_05130_amd as ie
from oracle import controller as O

EMERG, RECOV, CONT, NONE = O.EMERGENCY, O.RECOVERY, O.CONTENTION, O.NONE


def periods(ctl, obs):
    """obs: list of per-period lists of (kernels, klc) per instance -> tokens per period."""
    out = []
    for row in obs:
        for i, (k, t) in enumerate(row):
            ctl.report(i, k, t)
        out.append(ctl.issue())
    return out


# ------------------------------------------------------------------ oracle pins (paper text)
def test_alone_best_effort_gets_its_limit():
    # without an SLO-sensitive co-located instance the state stays NONE and the
    # instance runs at its limit, whatever it reports
    c = O.Controller()
    c.add(0.25, 0.75, False)
    for r in periods(c, [[(100, 5.0)], [(0, 0)], [(7, 9.0)]]):
        assert r == [256 * 0.75]
        assert c.state == NONE


def test_klc_violation_raises_emergency_and_shrinks_colocated():
    # a significant KLC increase of the SLO instance scales it up to its limit
    # at once; the co-located instance is scaled down by the KLC change
    c = O.Controller(eta_violation=0.2)
    c.add(0.5, 1.0, True)
    c.add(0.5, 0.75, False)
    r = periods(c, [[(85, 10.0), (85, 10.0)], [(85, 10.0), (85, 10.0)]])
    assert c.state == CONT and r[-1][0] == 128.0
    r_last = r[-1][1]
    c.report(0, 85, 15.0)            # KLC 10 -> 15 ms: dT = 0.5 > 0.2
    c.report(1, 85, 10.0)
    r = c.issue()
    assert c.state == EMERG
    assert r[0] == 256.0             # MaxTokens * limit
    assert r[1] == pytest.approx(min(128.0, r_last) * 10.0 / 15.0)   # scaled by T_min / T_current
    assert r[1] < r_last


def test_small_klc_change_is_contention():
    c = O.Controller(eta_violation=0.2)
    c.add(0.5, 1.0, True)
    c.add(0.5, 1.0, False)
    periods(c, [[(85, 10.0), (85, 10.0)]])
    r = periods(c, [[(85, 11.9), (85, 10.0)]] * 3)
    assert c.state == CONT
    assert r[-1][0] == 128.0                     # back at the request
    assert r[-1][1] == r[0][1] == r[1][1]       # CONTENTION keeps R_last


def test_only_the_raiser_leaves_emergency():
    # two SLO instances: A raises EMERGENCY; B's calm reading does not reset it;
    # once A's KLC recovers, A resets the state
    c = O.Controller(eta_violation=0.2)
    c.add(0.25, 1.0, True)
    c.add(0.25, 1.0, True)
    periods(c, [[(10, 10.0), (10, 10.0)]])
    periods(c, [[(10, 20.0), (10, 10.0)]])
    assert c.state == EMERG and c.owner == 0
    periods(c, [[(10, 20.0), (10, 10.0)]])
    assert c.state == EMERG
    r = periods(c, [[(10, 10.0), (10, 10.0)]])[-1]
    assert c.state == CONT and c.owner == -1
    assert r == [64.0, 64.0]


def test_idle_slo_instance_scales_down_and_colocated_grows():
    # no kernels from the SLO instance for a whole window: it drops to its
    # request, and the co-located instance grows by eta_increase per period up
    # to its limit
    c = O.Controller(window=3, eta_increase=1.25)
    c.add(0.25, 1.0, True)
    c.add(0.25, 0.5, False)
    rs = periods(c, [[(0, 0), (50, 10.0)]] * 8)
    assert all(r[0] == 64.0 for r in rs)
    assert c.state == RECOV
    grow = [r[1] for r in rs]
    expect, v = [], 64.0
    for _ in rs:
        v = min(v * 1.25, 128.0)
        expect.append(v)
    assert grow == expect
    assert grow[-1] == 128.0


def test_idle_after_a_violation_leaves_emergency_and_scales_down():
    # a burst raises EMERGENCY; when the SLO instance then goes quiet (no
    # kernels, no completed iteration) nothing is seen to slow down: it falls
    # back to its request at once and, after a whole idle window, the
    # co-located instance grows again (Sec. 3.4.1: no recent kernels -> scale
    # down).  A KLC held over from the burst would keep EMERGENCY and shrink
    # the neighbour by the KLC ratio every period instead.
    c = O.Controller(window=2, eta_violation=0.2, eta_increase=1.25)
    c.add(0.25, 0.5, True)
    c.add(0.75, 1.0, False)
    periods(c, [[(50, 10.0), (50, 10.0)]])
    r = periods(c, [[(50, 30.0), (50, 10.0)]])[-1]
    assert c.state == EMERG and r == [128.0, 192.0 / 3.0]
    rs, states = [], []
    for _ in range(5):
        rs.append(periods(c, [[(0, 0), (50, 10.0)]])[-1])
        states.append(c.state)
    assert states == [CONT, RECOV, RECOV, RECOV, RECOV]
    assert all(r[0] == 64.0 for r in rs)
    v, grow = 192.0 / 3.0, []
    for st in states:
        v = v if st == CONT else min(v * 1.25, 256.0)
        grow.append(v)
    assert [r[1] for r in rs] == grow


def test_listing_yield_persists_under_contention():
    # the listing: the yielded issue becomes R_last, and CONTENTION keeps it,
    # so while the SLO instance stays busy the co-located one stays shrunk;
    # two EMERGENCY periods in a row divide twice
    c = O.Controller(eta_violation=0.2)
    c.add(0.25, 0.5, True)
    c.add(0.75, 1.0, False)
    periods(c, [[(50, 10.0), (50, 10.0)]])
    r = periods(c, [[(50, 20.0), (50, 10.0)]] * 2 + [[(50, 10.0), (50, 10.0)]] * 3)
    assert [x[1] for x in r] == [96.0, 48.0, 48.0, 48.0, 48.0]
    assert [x[0] for x in r] == [128.0, 128.0, 64.0, 64.0, 64.0]


def test_temporary_yield_restores_the_plan():
    # the text's "temporarily resized down": the yield is taken from the plan
    # held before the emergency, does not compound, and CONTENTION restores it
    c = O.Controller(eta_violation=0.2, temporary_yield=True)
    c.add(0.25, 0.5, True)
    c.add(0.75, 1.0, False)
    periods(c, [[(50, 10.0), (50, 10.0)]])
    r = periods(c, [[(50, 20.0), (50, 10.0)]] * 2 + [[(50, 10.0), (50, 10.0)]] * 3)
    assert [x[1] for x in r] == [96.0, 96.0, 192.0, 192.0, 192.0]
    assert [x[0] for x in r] == [128.0, 128.0, 64.0, 64.0, 64.0]
    # once the SLO instance has been idle for a whole window (4 periods),
    # RECOVERY grows the co-located one from the plan, not from the yield
    r = periods(c, [[(0, 0), (50, 10.0)]] * 5)
    assert [x[1] for x in r] == [192.0, 192.0, 192.0, 240.0, 256.0]
    assert c.state == RECOV


def test_window_remembers_recent_kernels():
    # one burst keeps an instance active for exactly `window` periods
    c = O.Controller(window=3)
    c.add(0.25, 1.0, True)
    c.add(0.25, 1.0, False)
    states = []
    for row in [[(10, 5.0), (10, 5.0)]] + [[(0, 0), (10, 5.0)]] * 4:
        periods(c, [row])
        states.append(c.state)
    assert states == [CONT, CONT, CONT, RECOV, RECOV]


def test_idle_colocated_lets_slo_instance_grow_to_the_device():
    c = O.Controller(eta_increase=1.5)
    c.add(0.25, 0.5, True)
    c.add(0.25, 0.5, False)
    rs = periods(c, [[(20, 5.0), (0, 0)]] * 6)
    got = [r[0] for r in rs]
    v, expect = 64.0, []
    for _ in rs:
        v = min(v * 1.5, 256.0)                 # not capped at its limit (only at the device)
        expect.append(v)
    assert got == expect and got[-1] == 256.0


def test_tokens_to_disjoint_placements():
    c = O.Controller()
    for _ in range(4):
        c.add(0.25, 0.5, False)
    q, f = c.quotas([63.9, 100.0, 3.0, 43.0])   # 63.9 -> 64, 12.5 granules -> 13, min 8, 5.4 -> 5
    assert q == [64, 104, 8, 40]
    assert f == [192, 88, 80, 40]                 # best effort: downward from the top, id order


def cu_sets(q, f):
    return [set((fi + k) % 256 for k in range(qi)) for qi, fi in zip(q, f)]


def test_oversubscribed_placements_never_share_a_cu():
    # SLO-sensitive instances upward from bit 0; best-effort instances scaled
    # into the CUs left free, downward from the top
    c = O.Controller()
    c.add(0.25, 1.0, True)
    c.add(0.25, 0.5, False)
    c.add(0.25, 0.5, True)
    c.add(0.25, 0.5, False)
    q, f = c.quotas([128.0, 128.0, 64.0, 64.0])
    assert q == [128, 40, 64, 16]                  # 8 each + (120, 56) * 48 // 176 = (32, 15) -> 32, 8
    assert f == [0, 216, 128, 200]
    sets = cu_sets(q, f)
    assert all(not (sets[a] & sets[b]) for a in range(4) for b in range(a + 1, 4))
    # SLO tokens alone exceed the device: they give way so each best-effort
    # instance keeps min_quota, still without sharing
    q, f = c.quotas([256.0, 128.0, 200.0, 64.0])
    assert q[0] + q[2] <= 256 - 2 * 8 and min(q[1], q[3]) >= 8
    assert sum(q) <= 256
    sets = cu_sets(q, f)
    assert all(not (sets[a] & sets[b]) for a in range(4) for b in range(a + 1, 4))


@pytest.mark.parametrize("seed", range(20))
def test_random_placements_never_share_a_cu(seed):
    rng = np.random.default_rng(seed)
    c = O.Controller(granule=int(rng.choice([8, 32])), min_quota=32)
    n = int(rng.integers(1, 8))
    for _ in range(n):
        c.add(0.25, 1.0, bool(rng.random() < 0.5))
    q, f = c.quotas([float(v) for v in rng.uniform(0, 300, n)])
    assert all(32 <= x <= 256 for x in q)
    sets = cu_sets(q, f)
    assert all(not (sets[a] & sets[b]) for a in range(n) for b in range(a + 1, n))


# ------------------------------------------------------------------ library vs oracle
def random_scenario(seed, n_periods=300):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 5))
    insts = []
    for _ in range(n):
        req = float(rng.choice([0.125, 0.25, 0.5]))
        lim = float(min(1.0, req * rng.choice([1.0, 1.5, 2.0, 4.0])))
        insts.append((req, lim, bool(rng.random() < 0.5)))
    obs = []
    klc = [float(rng.uniform(1, 20)) for _ in range(n)]
    for _ in range(n_periods):
        row = []
        for i in range(n):
            idle = rng.random() < 0.25
            k = 0 if idle else int(rng.integers(1, 400))
            klc[i] = max(0.5, klc[i] * float(rng.choice([0.9, 1.0, 1.05, 1.6])))
            row.append((k, 0.0 if idle else klc[i]))
        obs.append(row)
    return insts, obs


@pytest.mark.parametrize("seed", range(12))
def test_library_matches_oracle(seed):
    insts, obs = random_scenario(seed)
    params = dict(window=int(1 + seed % 5), eta_violation=[0.1, 0.2, 0.5][seed % 3],
                  eta_increase=[1.1, 1.25, 2.0][seed % 3], temporary_yield=seed % 2 == 1)
    o = O.Controller(**params)
    lib = ie.Controller(**params)
    for req, lim, slo in insts:
        assert o.add(req, lim, slo) == lib.add(req, lim, slo)
    seen_states = set()
    for row in obs:
        for i, (k, t) in enumerate(row):
            o.report(i, k, t)
            lib.report(i, k, t)
        want = o.issue()
        wq, wf = o.quotas(want)
        got, gq, gf = lib.issue()
        assert got == want                        # same fp64 steps: exact
        assert (gq, gf) == (wq, wf)
        assert lib.state() == o.state
        seen_states.add(o.state)
    lib.close()
    if any(s for _, _, s in insts) and not all(s for _, _, s in insts):
        assert len(seen_states) >= 2


def test_controller_abi_errors():
    p = ie.CtlParams()
    ie.lib().iefwd_ctl_params_init(ie.ctypes.byref(p))
    h = ie.ctypes.c_void_p()
    for field, bad, status in [("abi_version", 99, ie.EVERSION), ("window", 0, ie.EINVAL),
                               ("min_quota", 300, ie.EINVAL), ("eta_increase", 0.5, ie.EINVAL),
                               ("eta_violation", math.nan, ie.EINVAL), ("flags", 2, ie.EINVAL)]:
        q = ie.CtlParams.from_buffer_copy(p)
        setattr(q, field, bad)
        assert ie.lib().iefwd_ctl_create(ie.ctypes.byref(q), ie.ctypes.byref(h)) == status, field
        assert h.value is None
    c = ie.Controller()
    for req, lim in [(0.0, 0.5), (0.5, 0.25), (0.5, 1.5)]:
        with pytest.raises(ie.IefwdError):
            c.add(req, lim, True)
    c.add(0.25, 0.5, True)
    with pytest.raises(ie.IefwdError):
        c.report(1, 1, 1.0)                         # no such id
    t = (ie.ctypes.c_double * 2)()
    assert ie.lib().iefwd_ctl_issue(c._h, t, None, None, 2) == ie.EINVAL
    assert ie.lib().iefwd_ctl_destroy(None) == ie.OK
    c.close()
