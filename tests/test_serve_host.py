"""Host logic of the serving harness's paired policy (no GPU): the pairing,
the placements it can issue, and the order in which it prepares their
hardware queues."""
import pytest

from paper_2503_05130_amd import serve


class FakeInst:
    def __init__(self, log, idx):
        self.log, self.idx, self.cache = log, idx, None

    def set_stream_cache(self, n):
        self.cache = n

    def prepare_quota(self, q, first):
        self.log.append((self.idx, q, first))

    def set_quota(self, q, first):
        pass

    def submit(self, x):
        pass

    def wait(self):
        pass


class FakeServed:
    def __init__(self, log, idx, slo):
        self.inst, self.slo, self.pool, self.applied = FakeInst(log, idx), slo, [None], None


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
    assert all(s.inst.cache == k for s in served)
