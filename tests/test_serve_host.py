"""Host logic of the serving harness's paired policy (no GPU): the pairing,
the placements it can issue, and the order in which it prepares their
hardware queues."""
import pytest

from paper_2503_05130_amd import serve


class FakeInst:
    """A stream cache like the library's: an LRU of placements, the one in use
    never evicted; prepare_quota creates a queue (logged) only for a placement
    not already cached."""

    def __init__(self, log, idx, n_cu=256):
        self.log, self.idx, self.cache = log, idx, 2
        self.current, self.pending = (n_cu, 0), None
        self.lru = [self.current]               # least recently used first

    def _touch(self, pl):
        if pl in self.lru:
            self.lru.remove(pl)
        else:
            self.log.append((self.idx,) + pl)
        self.lru.append(pl)
        self._trim()

    def _trim(self):
        while len(self.lru) > self.cache:
            victim = next(p for p in self.lru if p != self.current)
            self.lru.remove(victim)

    def set_stream_cache(self, n):
        self.cache = n
        self._trim()

    def prepare_quota(self, q, first):
        self._touch((q, first))

    def set_quota(self, q, first):
        self.pending = (q, first)

    def submit(self, x):
        if self.pending is not None:
            self.current, self.pending = self.pending, None
            self._touch(self.current)

    def wait(self):
        pass


class FakeServed:
    def __init__(self, log, idx, slo):
        self.inst, self.slo, self.pool, self.applied = FakeInst(log, idx), slo, [None], None

    def touch(self):
        self.inst.submit(None)


def mix(log):
    # the default mix's order: two SLO-sensitive encoders, then two best-effort decoders
    return [FakeServed(log, 0, True), FakeServed(log, 1, True), FakeServed(log, 2, False), FakeServed(log, 3, False)]


def test_pairs_and_placements():
    served = mix([])
    assert serve.pairs_of(served) == [(0, 2), (1, 3)]
    for pi in range(2):
        for sp in serve.PAIR_SPLITS:
            a = serve.paired_placement(256, pi, sp, False)
            b = serve.paired_placement(256, pi, sp, True)
            assert a[0] + b[0] == 128 and serve.placements_disjoint(a, b, 256)
            # the two pairs' regions never meet
            other = serve.paired_placement(256, 1 - pi, 64, False)
            assert serve.placements_disjoint(a, other, 256) and serve.placements_disjoint(b, other, 256)


def test_one_pair_owns_the_device():
    # one SLO-sensitive instance beside one best-effort one (inference beside
    # training): the pair's region is every CU, split in quarters
    assert serve.pair_region(256, 1) == 256 and serve.pair_region(256, 2) == 128
    assert serve.pair_region(256, 3) == 64
    got = [(serve.paired_placement(256, 0, sp, False, 256), serve.paired_placement(256, 0, sp, True, 256))
           for sp in serve.PAIR_SPLITS]
    assert got == [((64, 0), (192, 64)), ((128, 0), (128, 128)), ((192, 0), (64, 192))]
    for a, b in got:
        assert a[0] + b[0] == 256 and serve.placements_disjoint(a, b, 256)


@pytest.mark.parametrize("order", ["rounds", "instance"])
def test_prepare_order(monkeypatch, order):
    monkeypatch.setattr(serve.ie, "device_info", lambda dev: (256, 8))
    log = []
    served = mix(log)
    serve.prepare_paired(served, order)
    n, k = len(served), len(serve.PAIR_SPLITS)
    assert len(log) == n * k
    # every placement each instance can be given is prepared, once
    pairs = dict(serve.pairs_of(served))
    for idx in range(n):
        pi = 0 if idx in (0, 2) else 1
        second = idx not in pairs
        want = {serve.paired_placement(256, pi, sp, second) for sp in serve.PAIR_SPLITS}
        assert {(q, f) for i, q, f in log if i == idx} == want
    if order == "rounds":
        # the j-th queue made is instance j mod n's: each instance's queues share a residue
        assert [i for i, _, _ in log] == list(range(n)) * k
    else:
        assert [i for i, _, _ in log] == [i for i in range(n) for _ in range(k)]
    # the caches end holding exactly the prepared placements
    assert all(s.inst.cache == k and len(s.inst.lru) == k for s in served)


def test_prepare_rounds_after_another_policy(monkeypatch):
    # an earlier static policy left each instance's 64-CU placement cached; two
    # of them coincide with paired placements.  The rounds must still create
    # every placement, one queue per instance per round.
    monkeypatch.setattr(serve.ie, "device_info", lambda dev: (256, 8))
    log = []
    served = mix(log)
    for i, s in enumerate(served):
        s.inst.set_quota(64, 64 * i)
        s.inst.submit(None)
        s.inst.set_quota(256, 0)
        s.inst.submit(None)
    log.clear()
    assert {(64, 0), (64, 192)} & {serve.paired_placement(256, pi, 64, sec) for pi in (0, 1) for sec in (0, 1)}
    serve.prepare_paired(served, "rounds")
    k = len(serve.PAIR_SPLITS)
    assert [i for i, _, _ in log] == list(range(len(served))) * k


@pytest.mark.parametrize("cv", [1.0, 2.0, 4.0, 6.0])
def test_arrival_gaps_mean_and_cv(cv):
    # Gamma gaps with shape 1/cv^2 and scale cv^2/rate: mean 1/rate, std cv/rate
    import numpy as np
    g = serve.arrival_gaps(np.random.default_rng(7), 200.0, cv, 400_000)
    assert (g >= 0).all()
    assert abs(g.mean() * 200.0 - 1.0) < 0.03
    assert abs(g.std() / g.mean() - cv) < 0.03 * cv


def test_arrival_gaps_poisson_stream_unchanged():
    # cv 1 is the exponential stream the harness drew before the option existed
    import numpy as np
    a = serve.arrival_gaps(np.random.default_rng(5100), 200.0, 1.0, 1000)
    b = np.random.default_rng(5100).exponential(1.0 / 200.0, size=1000)
    assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        serve.arrival_gaps(np.random.default_rng(0), 200.0, 0.0, 4)


class FakeDev:
    """Stands in for an instance: every batch takes `ms` of device time."""

    def __init__(self, ms):
        self.ms, self.n = ms, 0

    def set_quota(self, q, first):
        pass

    def submit(self, x):
        self.n += 1

    def wait(self):
        import time
        time.sleep(self.ms / 1e3)

    def last_batch_ms(self):
        return self.ms

    def kernels_launched(self):
        return 100 * self.n


@pytest.mark.parametrize("klc", ["device", "cycle"])
def test_dispatcher_klc_modes(monkeypatch, klc):
    # a burst of 12 requests at t = 0 into batches of up to 4 taking 2 ms each:
    # device-time ratios stay 1, cycle ratios grow with the wait in the queue
    import threading
    import time
    import numpy as np
    monkeypatch.setattr(serve.ie, "device_info", lambda dev: (256, 8))
    s = object.__new__(serve.Served)
    s.idx, s.name, s.max_batch, s.rate, s.slo = 0, "fake", 4, 1.0, True
    s.inst, s.pool, s.lock, s.klc = FakeDev(2.0), [None] * 16, threading.Lock(), klc
    s.reset(1.0)
    s.arrivals = np.zeros(12)
    s.latency = np.full(12, np.nan)
    s.run(time.perf_counter(), 1.0, threading.Event())
    assert s.next == 12 and s.batches == 3 and np.isfinite(s.latency).all()
    if klc == "device":
        assert s.ratios == [1.0, 1.0, 1.0]
    else:
        # the k-th batch's oldest request waited for the k-1 batches before it
        assert all(r >= k + 1 for k, r in enumerate(s.ratios))
        assert s.ratios == sorted(s.ratios)


def test_serve_report_tables(capsys, tmp_path):
    # the report reads the harness's JSON lines: one row per instance result,
    # figures that do not apply shown as "-", the summary line echoed
    import json
    from paper_2503_05130_amd import serve_report
    res = {"policy": "alg2", "label": "alg2@100", "mean_quota": [64.0, 192.0],
           "state_counts": {"1": 2, "3": 8},
           "instances": [{"name": "bert_inf", "p50_ms": 0.9, "p95_ms": 1.4, "p99_ms": 1.7, "quota_changes": 3},
                         {"name": "bert_train", "training": True, "steps_s": 94.0, "quota_changes": 1}]}
    f = tmp_path / "out.jsonl"
    f.write_text(json.dumps({"setup_s": 1.0}) + "\n" + json.dumps(res) + "\n" +
                 json.dumps({"train_inf_summary": {"alg2": {"x": 1}}}) + "\n")
    assert serve_report.main([str(f)]) == 0
    out = capsys.readouterr().out.splitlines()
    assert out[0].startswith("| policy | instance |")
    assert out[2] == "| alg2@100 | bert_inf | 64.0 | 0.9 | 1.4 | 1.7 | - | - | 3 | EMERGENCY 2, CONTENTION 8 |"
    assert out[3] == "| alg2@100 | bert_train | 192.0 | - | - | - | 94.0 | - | 1 | EMERGENCY 2, CONTENTION 8 |"
    assert out[-1].startswith("train_inf_summary: ")
