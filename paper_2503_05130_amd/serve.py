"""Co-located serving on one GPU: Poisson or Gamma request streams into several
instances, one dispatcher thread per instance, and a quota policy that
re-masks the instances every control period (the paper's setting of
Sec. 3.4 and its inference-inference experiments, Sec. 5).

  python -m paper_2503_05130_amd.serve [--policy alg2 alg2@100 alg2p static proportional shared paired]
                                       [--horizon 20] [--warmup 2] [--period-ms 20] [--granule 32] [--small]
                                       [--mix inference|train|train2|decode] [--queue-probe]
                                       [--queue-order rounds|instance] [--cv 1] [--klc device|cycle]
                                       [--eta-violation 0.2] [--window 4] [--temporary-yield] [--timeline]
                                       [--exclusive]

Default mix: two BERT-base-shaped encoders (post-LN, 12 x 768, S = 128,
batches of up to 4, 200 requests/s each, latency-sensitive) and two causal
pre-LN decoders (24 x 2048, 16 heads, FFN 8192, S = 1024, batches of up to
2, 10 requests/s each, best effort).  Every request is one sequence; a
dispatcher takes up to `max_batch` requests that have arrived, runs them as
one batch and records each request's latency (completion - arrival).
Other mixes (--mix): train, that BERT-base-shaped encoder beside a training
instance of the same shape (Sec. 5 train-inf collocation); train2, two such
training instances (training-training collocation); decode, the encoder
beside a d = 2048 decoder generating token by token over its KV cache.  Each
of these also runs every instance alone on the whole GPU (exclusive), as
--exclusive does for the default mix.

Policies (each period):
  shared       every instance on all CUs (no partitioning)
  static       each instance on its request share, disjoint
  proportional quota proportional to the queue length (multiples of 32
               CUs, at least 32), disjoint, all CUs handed out
  alg2         the fast scale-up/down controller (iefwd_ctl_*, 32-CU
               granule): kernels launched in the period and the per-batch
               time go in, quotas and placements come out.  A placement's
               queue is made when the placement is first issued, in
               whatever order the controller issues them, so the creation
               order described under paired is not kept
  alg2p        Alg. 2 on the paired policy's placements: the controller
               issues quotas as under alg2, and each pair's region is split
               in the ratio of its two members' quotas, to the nearest of
               the prepared splits (queues made as under paired)
  paired       quotas from a fixed vocabulary: instances are paired (each
               SLO-sensitive one with a best-effort one) and each pair owns
               a fixed region (the CUs split evenly among the pairs: 128 for
               two pairs, all 256 for one) whose split point moves in
               quarters of the region (32 / 96, 64 / 64, 96 / 32 of 128) in
               proportion to the two queue lengths (a training instance
               counts as one queued request).  Every placement is prepared before the run and the
               stream caches hold all of them, so no hardware queue is
               created or destroyed while the instances serve (creating or
               destroying one stalls every queue of the process for ~3 ms on
               MI355X, and more than ~20-24 live queues per process make the
               hardware scheduler time-slice them).  The placements are
               prepared in rounds, one queue per instance per round, in the
               order the instances made their first queues (--queue-order
               rounds); --queue-order instance prepares each instance's
               placements in turn.  Measured on MI355X: in round order an
               encoder's batches are unaffected by the decoders' long GEMM
               launches; in instance order they run 5-8 x slower while any
               decoder GEMM runs, whichever CUs it runs on.  This fits the
               queues being dealt to the hardware's dispatch pipes in
               creation order, with a queue waiting behind a neighbour's
               launch whose workgroups are still being placed on the same
               pipe.

--granule sets the quota granularity (in CUs) of proportional and alg2.

--cv sets the coefficient of variation of the inference instances'
inter-arrival gaps: 1 is a Poisson stream; other values draw Gamma-distributed
gaps of the same mean (shape 1/cv^2), the fluctuating workloads of the paper's
fast-adaptivity experiment (Sec. 5).  In the train and decode mixes it applies
to the inference instance.

A new quota's masked stream is created by the control thread
(iefwd_prepare_quota_at) before the quota is posted, so a dispatcher only
switches streams at its next batch boundary.

The KLC an instance reports for a period is the median, over the batches it
completed in the period, of each batch's device time relative to the fastest
batch of the same size it has run on the same quota (times 1 ms).  So the
controller's KLC change measures the slowdown of an iteration of one shape on
one CU share -- contention -- rather than a change of batch size or of its own
quota (which the controller itself causes).  This per-<batch, quota> baseline
is what the paper's profiler supplies (Sec. 3.2).

--timeline adds to each policy's result, per control period, its end time,
the quotas posted, the controller state and the requests that arrived at each
inference instance.

--klc cycle measures instead each batch's cycle from the arrival of its oldest
request to its completion, relative to the same fastest device time.  The
paper reads a KLC rise as contention or a burst of the instance's own requests
(Sec. 3.4.1); there an instance's kernels wait for tokens, so a burst
lengthens its launch cycle.  Under CU masks nothing holds a launch back and a
batch's device time does not see a burst, which shows only as requests
waiting for the instance's CUs: the cycle counts that wait.

Inputs are seeded synthetic embeddings already in device memory; weights are
the library's seeded random init.
"""
from __future__ import annotations

import argparse
import json
import threading
import time

import numpy as np
import torch

import paper_2503_05130_amd as ie

BERT = dict(n_layers=12, d_model=768, n_heads=12, d_ff=3072, pre_ln=0, causal=0, n_out=2)
DECODER = dict(n_layers=24, d_model=2048, n_heads=16, d_ff=8192, pre_ln=1, causal=1, n_out=2)
SMALL = dict(n_layers=2, d_model=256, n_heads=4, d_ff=1024, pre_ln=0, causal=0, n_out=2)


def default_mix(small: bool = False):
    """(name, shape, seq, max_batch, rate/s, request, limit, slo_sensitive, weight seed)."""
    if small:
        return [("enc_a", SMALL, 64, 4, 200.0, 0.25, 0.5, True, 51),
                ("enc_b", SMALL, 64, 4, 200.0, 0.25, 0.5, True, 52),
                ("dec_a", dict(SMALL, pre_ln=1, causal=1), 256, 2, 20.0, 0.25, 0.5, False, 53),
                ("dec_b", dict(SMALL, pre_ln=1, causal=1), 256, 2, 20.0, 0.25, 0.5, False, 54)]
    return [("bert_a", BERT, 128, 4, 200.0, 0.25, 0.5, True, 51),
            ("bert_b", BERT, 128, 4, 200.0, 0.25, 0.5, True, 52),
            ("dec_a", DECODER, 1024, 2, 10.0, 0.25, 0.5, False, 53),
            ("dec_b", DECODER, 1024, 2, 10.0, 0.25, 0.5, False, 54)]


def arrival_gaps(rng, rate, cv, n):
    """n inter-arrival gaps of mean 1/rate.  cv 1: exponential (a Poisson
    stream); otherwise Gamma with shape 1/cv^2 and scale cv^2/rate, whose
    coefficient of variation is cv -- the fluctuating workloads of the paper's
    fast-adaptivity experiment (Sec. 5), where CV grows up to 6."""
    if cv <= 0:
        raise ValueError("cv must be positive")
    if cv == 1.0:
        return rng.exponential(1.0 / rate, size=n)
    k = 1.0 / (cv * cv)
    return rng.gamma(k, 1.0 / (rate * k), size=n)


class Served:
    """One instance with its request stream, pool of inputs and statistics."""

    cv = 1.0                                # coefficient of variation of the inter-arrival gaps
    klc = "device"                          # what the KLC of a batch measures: "device" or "cycle"

    def __init__(self, idx, name, shape, seq, max_batch, rate, request, limit, slo, seed, pool=16):
        self.idx, self.name, self.seq, self.max_batch, self.rate = idx, name, seq, max_batch, rate
        self.request, self.limit, self.slo = request, limit, slo
        self.inst = ie.Instance(device=0, max_batch=max_batch, max_seq=seq, seed=seed, **shape)
        rng = np.random.default_rng(5000 + idx)
        d = shape["d_model"]
        self.pool = torch.from_numpy(rng.standard_normal((pool, seq, d), dtype=np.float32)).to("cuda:0")
        self.lock = threading.Lock()

    def reset(self, horizon):
        """Fresh request stream (the same for every policy) and statistics."""
        arr = np.random.default_rng(5100 + self.idx)
        gaps = arrival_gaps(arr, self.rate, self.cv, int(self.rate * horizon * 2) + 16)
        t = np.cumsum(gaps)
        self.arrivals = t[t < horizon]
        self.latency = np.full(len(self.arrivals), np.nan)
        self.next = 0                       # first request not yet dispatched
        self.best_ms = {}                   # fastest batch time per (batch size, quota)
        self.kernels = self.inst.kernels_launched()   # read by the control thread
        self.ratios = []                    # batch time / best, batches of the current period
        self.pending = None                 # (quota, first) posted by the control thread
        self.inst.set_quota(ie.device_info(0)[0], 0)
        self.applied = (ie.device_info(0)[0], 0)
        self.busy = False                   # a batch is in flight (on `applied`)
        self.batch_log = []                 # (completion time, device ms, quota, first batch after a switch)
        self.batches = 0
        self.changes = 0                    # quota switches applied
        self.klc_log = []                   # KLC ratios reported to the controller
        self.plans = set()                  # distinct (quota, first) applied

    def queue_len(self, now):
        return int(np.searchsorted(self.arrivals, now, side="right")) - self.next

    def touch(self):
        """One small batch, so that a posted quota takes effect."""
        self.inst.submit(self.pool[:1])
        self.inst.wait()

    def run(self, t0, horizon, stop):
        slot = 0
        while not stop.is_set():
            now = time.perf_counter() - t0
            if self.next >= len(self.arrivals) or now > horizon + 5.0:
                return
            if self.arrivals[self.next] > now:
                time.sleep(min(self.arrivals[self.next] - now, 0.002))
                continue
            k = min(self.max_batch, self.queue_len(now))
            oldest = self.arrivals[self.next]
            with self.lock:                 # taking the quota and marking the batch start together
                pend, self.pending = self.pending, None
                self.busy = True
            switched = pend is not None and pend != self.applied
            if switched:
                self.inst.set_quota(*pend)
                self.changes += 1
                self.plans.add(pend)
            with self.lock:
                if pend is not None:
                    self.applied = pend
            x = self.pool[slot:slot + k]
            slot = (slot + k) % (len(self.pool) - self.max_batch + 1)
            self.inst.submit(x)
            self.inst.wait()
            with self.lock:
                self.busy = False
            done = time.perf_counter() - t0
            self.latency[self.next:self.next + k] = done - self.arrivals[self.next:self.next + k]
            self.next += k
            self.batches += 1
            ms = self.inst.last_batch_ms()
            self.batch_log.append((done, ms, self.applied[0] if self.applied else 0, switched))
            key = (k, self.applied[0] if self.applied else 0)
            best = min(self.best_ms.get(key, ms), ms)
            self.best_ms[key] = best
            cyc = (done - oldest) * 1e3 if self.klc == "cycle" else ms
            with self.lock:
                self.kernels = self.inst.kernels_launched()
                self.ratios.append(cyc / best)

    def batch_stats(self, warmup):
        """Device time per batch (ms): first batches after a quota switch and the others."""
        log = [b for b in self.batch_log if b[0] >= warmup]
        out = {}
        for key, sel in (("after_switch", [b[1] for b in log if b[3]]), ("other", [b[1] for b in log if not b[3]])):
            if sel:
                out[key] = {"n": len(sel), "p50_ms": round(float(np.percentile(sel, 50)), 3),
                            "p99_ms": round(float(np.percentile(sel, 99)), 3), "max_ms": round(float(max(sel)), 3)}
        return out

    def stats(self, warmup):
        keep = (self.arrivals >= warmup) & np.isfinite(self.latency)
        lat = self.latency[keep] * 1e3
        return {"name": self.name, "requests": int(keep.sum()), "dropped": int(np.isnan(self.latency).sum()),
                "batch_device_ms": self.batch_stats(warmup),
                "p50_ms": round(float(np.percentile(lat, 50)), 3) if len(lat) else None,
                "p95_ms": round(float(np.percentile(lat, 95)), 3) if len(lat) else None,
                "p99_ms": round(float(np.percentile(lat, 99)), 3) if len(lat) else None,
                "batches": self.batches, "quota_changes": self.changes, "distinct_placements": len(self.plans),
                "klc_ratio_p50_p90": ([round(float(np.percentile(self.klc_log, p)), 3) for p in (50, 90)]
                                      if self.klc_log else None)}


class Trainee:
    """A training instance co-located with inference (the paper's train-inf
    collocation, Sec. 5.2): whole training steps back to back on a fixed
    synthetic batch, with the same quota hand-off and controller reports as
    an inference instance.  Its KLC is the step time relative to its fastest
    step on the same quota; it always has work, so its queue length is 1."""

    def __init__(self, idx, name, shape, seq, batch, request, limit, seed):
        self.idx, self.name, self.seq, self.max_batch, self.rate = idx, name, seq, batch, 0.0
        self.request, self.limit, self.slo = request, limit, False
        self.inst = ie.Trainer(device=0, max_batch=batch, max_seq=seq, seed=seed, **shape)
        self.x = torch.from_numpy(np.random.default_rng(6000 + idx).standard_normal(
            (batch, seq, shape["d_model"]), dtype=np.float32)).to("cuda:0")
        self.labels = torch.from_numpy(np.random.default_rng(6100 + idx).integers(
            0, shape["n_out"], size=(batch, seq), dtype=np.int32)).to("cuda:0")
        self.pool = self.x
        self.lock = threading.Lock()

    def reset(self, horizon):
        self.done_at = []                   # completion times of the steps
        self.step_ms = []
        self.best_ms = {}
        self.kernels = self.inst.kernels_launched()
        self.ratios = []
        self.pending = None
        self.inst.set_quota(ie.device_info(0)[0], 0)
        self.applied = (ie.device_info(0)[0], 0)
        self.busy = False                   # a step is in flight (on `applied`)
        self.batches = 0
        self.changes = 0
        self.klc_log = []
        self.plans = set()

    def queue_len(self, now):
        return 1

    def warm(self):
        self.inst.step(self.x, self.labels)
        self.inst.wait()

    touch = warm                            # one step applies a posted quota

    def run(self, t0, horizon, stop):
        while not stop.is_set():
            if time.perf_counter() - t0 > horizon:
                return
            with self.lock:
                pend, self.pending = self.pending, None
                self.busy = True
            if pend is not None and pend != self.applied:
                self.inst.set_quota(*pend)
                with self.lock:
                    self.applied = pend
                self.changes += 1
                self.plans.add(pend)
            self.inst.step(self.x, self.labels)
            self.inst.wait()
            with self.lock:
                self.busy = False
            self.done_at.append(time.perf_counter() - t0)
            ms = self.inst.last_batch_ms()
            self.step_ms.append(ms)
            self.batches += 1
            best = min(self.best_ms.get(self.applied[0], ms), ms)
            self.best_ms[self.applied[0]] = best
            with self.lock:
                self.kernels = self.inst.kernels_launched()
                self.ratios.append(ms / best)

    def stats(self, warmup, horizon):
        done = np.array(self.done_at)
        n = int(((done >= warmup) & (done <= horizon)).sum())
        return {"name": self.name, "training": True, "steps": n,
                "steps_s": round(n / max(horizon - warmup, 1e-9), 2),
                "sequences_s": round(n * self.max_batch / max(horizon - warmup, 1e-9), 1),
                "step_ms_p50": round(float(np.median(self.step_ms)), 3) if self.step_ms else None,
                "quota_changes": self.changes, "distinct_placements": len(self.plans),
                "klc_ratio_p50_p90": ([round(float(np.percentile(self.klc_log, p)), 3) for p in (50, 90)]
                                      if self.klc_log else None)}


class Generator:
    """A decoding instance co-located with inference (the decode phase beside
    prefill-type work): requests of a P-token prompt per sequence (one prefill
    batch) followed by G decode steps of one token per sequence, back to back,
    over a KV cache.  Every prefill and every decode step is an iteration: a
    pending quota is applied before it, and its KLC is its device time
    relative to the fastest iteration of the same kind on the same quota.  It
    always has work, so its queue length is 1."""

    def __init__(self, idx, name, shape, batch, prompt, gen, request, limit, slo, seed):
        self.idx, self.name, self.max_batch, self.rate = idx, name, batch, 0.0
        self.prompt, self.gen = prompt, gen
        self.request, self.limit, self.slo = request, limit, slo
        self.inst = ie.Instance(device=0, max_batch=batch, max_seq=prompt + gen, seed=seed, kv_cache=1, **shape)
        x = np.random.default_rng(7000 + idx).standard_normal((batch, prompt + gen, shape["d_model"]),
                                                              dtype=np.float32)
        self.x_prompt = torch.from_numpy(np.ascontiguousarray(x[:, :prompt])).to("cuda:0")
        self.x_steps = [torch.from_numpy(np.ascontiguousarray(x[:, prompt + g])).to("cuda:0") for g in range(gen)]
        self.pool = self.x_prompt
        self.lock = threading.Lock()

    def reset(self, horizon):
        self.step_done, self.step_ms = [], []      # decode steps: completion time, wall time
        self.prefill_ms = []
        self.best_ms = {}
        self.kernels = self.inst.kernels_launched()
        self.ratios = []
        self.pending = None
        self.inst.set_quota(ie.device_info(0)[0], 0)
        self.applied = (ie.device_info(0)[0], 0)
        self.busy = False                   # an iteration is in flight (on `applied`)
        self.batches = 0
        self.changes = 0
        self.klc_log = []
        self.plans = set()

    def queue_len(self, now):
        return 1

    def warm(self):
        self.inst.submit(self.x_prompt)
        self.inst.wait()
        self.inst.decode(self.x_steps[0], self.prompt)
        self.inst.wait()

    def touch(self):
        """One prefill, so that a posted quota takes effect."""
        self.inst.submit(self.x_prompt)
        self.inst.wait()

    def _iteration(self, kind, launch):
        with self.lock:
            pend, self.pending = self.pending, None
            self.busy = True
        if pend is not None and pend != self.applied:
            self.inst.set_quota(*pend)
            with self.lock:
                self.applied = pend
            self.changes += 1
            self.plans.add(pend)
        t = time.perf_counter()
        launch()
        self.inst.wait()
        with self.lock:
            self.busy = False
        wall = (time.perf_counter() - t) * 1e3
        ms = self.inst.last_batch_ms()
        self.batches += 1
        key = (kind, self.applied[0])
        best = min(self.best_ms.get(key, ms), ms)
        self.best_ms[key] = best
        with self.lock:
            self.kernels = self.inst.kernels_launched()
            self.ratios.append(ms / best)
        return wall

    def run(self, t0, horizon, stop):
        while not stop.is_set():
            if time.perf_counter() - t0 > horizon:
                return
            self.prefill_ms.append(self._iteration("prefill", lambda: self.inst.submit(self.x_prompt)))
            for g in range(self.gen):
                if stop.is_set() or time.perf_counter() - t0 > horizon:
                    return
                wall = self._iteration("decode", lambda: self.inst.decode(self.x_steps[g], self.prompt + g))
                self.step_done.append(time.perf_counter() - t0)
                self.step_ms.append(wall)

    def stats(self, warmup, horizon):
        done = np.array(self.step_done)
        keep = (done >= warmup) & (done <= horizon)
        tpot = np.array(self.step_ms)[keep] if len(done) else np.zeros(0)
        n = int(keep.sum())
        return {"name": self.name, "decoding": True, "steps": n,
                "tokens_s": round(n * self.max_batch / max(horizon - warmup, 1e-9), 1),
                "tpot_p50_ms": round(float(np.percentile(tpot, 50)), 3) if n else None,
                "tpot_p99_ms": round(float(np.percentile(tpot, 99)), 3) if n else None,
                "prefill_p50_ms": round(float(np.median(self.prefill_ms)), 3) if self.prefill_ms else None,
                "quota_changes": self.changes, "distinct_placements": len(self.plans),
                "klc_ratio_p50_p90": ([round(float(np.percentile(self.klc_log, q)), 3) for q in (50, 90)]
                                      if self.klc_log else None)}


GRANULE = 32   # default quota granularity of the dynamic policies: 4 CUs per XCD, few distinct masks
PAIR_SPLITS = (32, 64, 96)   # first instance's share of its pair's region, in 128ths


def pair_region(n_cu, n_pairs):
    """CUs each pair owns: the device split evenly, in multiples of 32."""
    return max(32, (n_cu // max(n_pairs, 1)) // 32 * 32)


def pairs_of(served):
    """(first, second) index pairs for the paired policy: each SLO-sensitive
    instance with a best-effort one, in order; leftovers pair among themselves."""
    slo = [i for i, s in enumerate(served) if s.slo]
    other = [i for i, s in enumerate(served) if not s.slo]
    pairs = list(zip(slo, other))
    rest = slo[len(pairs):] + other[len(pairs):]
    pairs += list(zip(rest[0::2], rest[1::2]))
    return pairs


def placements_disjoint(p, q, n_cu):
    """Whether two (quota, first bit) runs of mask bits share no CU."""
    bits = lambda r: {(r[1] + i) % n_cu for i in range(r[0])}
    return not (bits(p) & bits(q))


def paired_placement(n_cu, pair_idx, split, second, region=128):
    """(quota, first bit) of one member of pair `pair_idx` at a given split
    (PAIR_SPLITS: 128ths of the pair's `region` CUs)."""
    base = (region * pair_idx) % n_cu
    cut = split * region // 128
    return (region - cut, base + cut) if second else (cut, base)


def controller_quotas(ctl, served, last_k, firsts_out=None):
    """One Alg. 2 period: reports each instance's kernels launched and KLC
    (the median batch-time ratio of the period), returns the issued quotas
    (and appends the issued first mask bits to firsts_out)."""
    for i, s in enumerate(served):
        with s.lock:
            k, ratios = s.kernels, s.ratios
            s.ratios = []
        klc = float(np.median(ratios)) if ratios else 0.0
        if klc > 0:
            s.klc_log.append(klc)
        ctl.report(i, k - last_k[i], klc)
        last_k[i] = k
    _, qs, firsts = ctl.issue()
    if firsts_out is not None:
        firsts_out.extend(firsts)
    return list(qs)


def control_loop(policy, served, t0, horizon, period, stop, history, granule=GRANULE, ctl_params=None):
    n_cu = ie.device_info(0)[0]
    ctl = None
    paired_like = policy in ("paired", "alg2p")
    if policy in ("alg2", "alg2p"):
        ctl = ie.Controller(max_tokens=n_cu, granule=granule, min_quota=granule, **(ctl_params or {}))
        for s in served:
            ctl.add(s.request, s.limit, s.slo)
    last_k = [s.kernels for s in served]
    posted = [s.applied if paired_like else None for s in served]
    while not stop.is_set():
        now = time.perf_counter() - t0
        if now > horizon:
            return
        if policy == "shared":
            plan = [(n_cu, 0)] * len(served)
        elif policy == "static":
            plan, first = [], 0
            for s in served:
                q = max(8, int(round(s.request * n_cu / 8)) * 8)
                plan.append((q, first))
                first = (first + q) % n_cu
        elif policy == "proportional":
            ql = np.array([max(s.queue_len(now), 0) for s in served], dtype=np.float64)
            share = np.full(len(served), 1.0 / len(served)) if ql.sum() == 0 else ql / ql.sum()
            qs = np.maximum(granule, np.floor(share * n_cu / granule) * granule).astype(int)
            while qs.sum() > n_cu:
                qs[int(np.argmax(qs))] -= granule
            qs[int(np.argmax(share))] += n_cu - qs.sum()
            plan, first = [], 0
            for q in qs:
                plan.append((int(q), first))
                first = (first + int(q)) % n_cu
        elif paired_like:
            # Hand-over in order: a member may shrink at once, but it grows only
            # onto CUs its partner has already left (the partner's current or
            # last batch ran on `applied`; a quota change takes effect at a batch
            # boundary, and a decoder batch runs for tens of ms).
            if policy == "alg2p":
                # Alg. 2 decides the quotas; each pair's region is split in the
                # ratio of its two members' quotas, to the nearest prepared split
                cq = controller_quotas(ctl, served, last_k)
            plan = list(posted)
            pairs = pairs_of(served)
            region = pair_region(n_cu, len(pairs))
            for pi, (a, b) in enumerate(pairs):
                if policy == "alg2p":
                    share = cq[a] / max(cq[a] + cq[b], 1)
                else:
                    la, lb = max(served[a].queue_len(now), 0), max(served[b].queue_len(now), 0)
                    share = 0.5 if la + lb == 0 else la / (la + lb)
                split = min(PAIR_SPLITS, key=lambda sp: abs(sp / 128.0 - share))
                want = {a: paired_placement(n_cu, pi, split, False, region),
                        b: paired_placement(n_cu, pi, split, True, region)}
                grow = [i for i in (a, b) if want[i][0] > posted[i][0]]
                for i in (a, b):                # the shrinking (or unchanged) member: posted at once
                    if i not in grow:
                        plan[i] = want[i]
                        with served[i].lock:
                            served[i].pending = want[i]
                for i in grow:                  # the growing one: once its partner has left the CUs
                    other = b if i == a else a
                    with served[other].lock:
                        held, busy = served[other].applied, served[other].busy
                    if not busy or placements_disjoint(want[i], held, n_cu):
                        plan[i] = want[i]
        else:
            firsts = []
            qs = controller_quotas(ctl, served, last_k, firsts)
            plan = list(zip(qs, firsts))
        # shrinking instances first, so that none starts a batch on CUs just handed to another
        order = sorted(range(len(served)), key=lambda i: plan[i][0] - (posted[i] or plan[i])[0])
        for i in order:
            s, p = served[i], plan[i]
            if p != posted[i]:
                if not paired_like:            # paired: every placement was prepared before the run
                    s.inst.prepare_quota(*p)   # hardware queue created here, not on the batch path
                posted[i] = p
            with s.lock:
                s.pending = p
        history.append((round(now, 3), [p[0] for p in plan], ctl.state() if ctl else -1))
        time.sleep(period)


def prepare_paired(served, queue_order="rounds"):
    """Prepares every placement the paired policy can issue, sizes each stream
    cache to hold exactly them (the full-device stream is dropped), and starts
    every instance on the even split.  Every cached masked stream but the
    full-device one is destroyed first, so that each placement is created
    here, in the chosen order.  queue_order "rounds": one new queue per
    instance per round, instances in the order their full-device queues were
    made, so that the k-th queue of every instance sits at the same position
    modulo the instance count; "instance": each instance's queues in turn."""
    n_cu = ie.device_info(0)[0]
    pairs = pairs_of(served)
    region = pair_region(n_cu, len(pairs))
    members = sorted((idx, pi, second) for pi, (a, b) in enumerate(pairs)
                     for idx, second in ((a, False), (b, True)))
    for idx, _, _ in members:
        # Only the full-device stream survives: a placement still cached from
        # an earlier policy would not be created below, and every later queue
        # would land one step off the round order.
        inst = served[idx].inst
        inst.set_quota(n_cu, 0)
        served[idx].touch()
        inst.set_stream_cache(1)
        inst.set_stream_cache(len(PAIR_SPLITS) + 1)
    if queue_order == "rounds":
        jobs = [(m, sp) for sp in PAIR_SPLITS for m in members]
    else:
        jobs = [(m, sp) for m in members for sp in PAIR_SPLITS]
    for (idx, pi, second), sp in jobs:
        served[idx].inst.prepare_quota(*paired_placement(n_cu, pi, sp, second, region))
    for idx, pi, second in members:
        inst = served[idx].inst
        start = paired_placement(n_cu, pi, 64, second, region)
        inst.set_quota(*start)
        served[idx].applied = start
        served[idx].touch()                 # moves the instance onto its placement
        inst.set_stream_cache(len(PAIR_SPLITS))


def run_policy(policy, served, horizon, warmup, period, granule=GRANULE, queue_order="rounds", ctl_params=None,
               timeline=False):
    for s in served:
        s.reset(horizon)
        if isinstance(s, (Trainee, Generator)):
            s.warm()
        else:
            s.inst.submit(s.pool[:1])          # warm the instance and its full-device stream
            s.inst.wait()
    if policy in ("paired", "alg2p"):
        prepare_paired(served, queue_order)
    torch.cuda.synchronize()
    stop, history = threading.Event(), []
    t0 = time.perf_counter()
    threads = [threading.Thread(target=s.run, args=(t0, horizon, stop)) for s in served]
    ctl = threading.Thread(target=control_loop,
                           args=(policy, served, t0, horizon, period, stop, history, granule, ctl_params))
    for t in threads + [ctl]:
        t.start()
    for t in threads:
        t.join()
    stop.set()
    ctl.join()
    qs = np.array([h[1] for h in history]) if history else np.zeros((0, len(served)))
    states = [h[2] for h in history]
    if policy in ("paired", "alg2p"):
        for s in served:
            s.inst.set_stream_cache(2)
    lat = [s.latency[(s.arrivals >= warmup) & np.isfinite(s.latency)] * 1e3 for s in served
           if isinstance(s, Served)]
    allat = np.concatenate(lat) if lat else np.zeros(0)
    aggregate = {"requests_s": round(len(allat) / max(horizon - warmup, 1e-9), 1),
                 "p50_ms": round(float(np.percentile(allat, 50)), 3) if len(allat) else None,
                 "p95_ms": round(float(np.percentile(allat, 95)), 3) if len(allat) else None,
                 "p99_ms": round(float(np.percentile(allat, 99)), 3) if len(allat) else None}
    extra = {"queue_order": queue_order} if policy in ("paired", "alg2p") else {}
    if policy in ("alg2", "alg2p") and ctl_params:
        extra["ctl_params"] = dict(ctl_params)
    if timeline:
        # per control period: its end (s), the quotas posted, the controller state
        # (-1 without one) and the requests that arrived at each instance in it
        ends = [h[0] for h in history]
        edges = np.array([0.0] + ends)
        arrived = [np.histogram(s.arrivals, bins=edges)[0].tolist() if isinstance(s, Served) and len(ends)
                   else [None] * len(ends) for s in served]
        extra["timeline"] = [[h[0], h[1], h[2], [a[i] for a in arrived]] for i, h in enumerate(history)]
    return {"policy": policy, **extra, "horizon_s": horizon, "warmup_s": warmup, "period_ms": period * 1e3,
            "granule": granule if policy in ("proportional", "alg2", "alg2p") else None, "aggregate": aggregate,
            "instances": [s.stats(warmup, horizon) if isinstance(s, (Trainee, Generator)) else s.stats(warmup)
                          for s in served],
            "mean_quota": [round(float(v), 1) for v in qs.mean(0)] if len(qs) else None,
            "periods": len(history),
            "state_counts": {str(k): states.count(k) for k in sorted(set(states))}}


def build_mix(mix):
    return [Served(i, *m) for i, m in enumerate(mix)]


def run_with_exclusive(served, policies, horizon, warmup, period, ctl_params=None, timeline=False):
    """Each policy with every instance ("label" keeps a policy's @period),
    then each instance alone on the whole GPU ("exclusive:<name>"); closes
    the instances.  Returns the results and the exclusive statistics by name."""
    out = []
    try:
        for pol in policies:
            name, _, per = pol.partition("@")
            res = run_policy(name, served, horizon, warmup, (float(per) if per else period) / 1e3,
                             ctl_params=ctl_params, timeline=timeline)
            res["label"] = pol
            out.append(res)
            print(json.dumps(res), flush=True)
        for one in served:
            res = run_policy("shared", [one], horizon, warmup, period / 1e3)
            res["policy"] = f"exclusive:{one.name}"
            out.append(res)
            print(json.dumps(res), flush=True)
    finally:
        for s in served:
            s.inst.close()
    excl = {r["instances"][0]["name"]: r["instances"][0] for r in out if r["policy"].startswith("exclusive")}
    return out, excl


def train_mix(small: bool = False):
    """The train-inf collocation mix: one BERT-base-shaped inference instance
    (batches of up to 4, latency-sensitive) beside one training instance of the
    same shape (batch 32 x 128, best effort)."""
    shape, seq = (SMALL, 64) if small else (BERT, 128)
    inf = Served(0, "bert_inf", shape, seq, 4, 200.0, 0.25, 0.5, True, 51)
    trn = Trainee(1, "bert_train", shape, seq, 8 if small else 32, 0.75, 1.0, 55)
    return [inf, trn]


def run_train_mix(policies, horizon, warmup, period, small=False, cv=1.0, klc="device", ctl_params=None,
                  timeline=False):
    """Each policy with both instances, then each instance alone on the whole
    GPU ("exclusive"); the paper compares co-location against exclusive."""
    served = train_mix(small)
    served[0].cv, served[0].klc = cv, klc   # the inference instance's arrivals and KLC
    out, excl = run_with_exclusive(served, policies, horizon, warmup, period, ctl_params, timeline)
    summary = {}
    for r in out:
        if r["policy"].startswith("exclusive"):
            continue
        inf, trn = r["instances"]
        e_inf, e_trn = excl["bert_inf"], excl["bert_train"]
        summary[r.get("label", r["policy"])] = {
            "inference_p50_vs_exclusive": round(inf["p50_ms"] / e_inf["p50_ms"], 3) if inf["p50_ms"] else None,
            "inference_p95_vs_exclusive": round(inf["p95_ms"] / e_inf["p95_ms"], 3) if inf["p95_ms"] else None,
            "inference_p99_vs_exclusive": round(inf["p99_ms"] / e_inf["p99_ms"], 3) if inf["p99_ms"] else None,
            "training_throughput_vs_exclusive": round(trn["steps_s"] / e_trn["steps_s"], 3) if e_trn["steps_s"] else None}
    print(json.dumps({"train_inf_summary": summary, "cv": cv, "klc": klc}), flush=True)
    return out, summary


def train2_mix(small: bool = False):
    """The training-training collocation mix (Sec. 5): two BERT-base-shaped
    training instances (batch 32 x 128 each, different seeds), both best
    effort, request 50% / limit 100%."""
    shape, seq, b = (SMALL, 64, 8) if small else (BERT, 128, 32)
    return [Trainee(0, "train_a", shape, seq, b, 0.5, 1.0, 55), Trainee(1, "train_b", shape, seq, b, 0.5, 1.0, 57)]


def run_train2_mix(policies, horizon, warmup, period, small=False, ctl_params=None, timeline=False):
    """Each policy with both training instances, then each alone.  The
    paper's figure of merit is the aggregate of the two throughputs, each
    normalised by its exclusive throughput (2.0 would be two exclusive GPUs'
    worth)."""
    served = train2_mix(small)
    out, excl = run_with_exclusive(served, policies, horizon, warmup, period, ctl_params, timeline)
    summary = {}
    for r in out:
        if r["policy"].startswith("exclusive"):
            continue
        fr = [st["steps_s"] / excl[st["name"]]["steps_s"] if excl[st["name"]]["steps_s"] else 0.0
              for st in r["instances"]]
        summary[r.get("label", r["policy"])] = {"throughput_vs_exclusive": [round(f, 3) for f in fr],
                                                "aggregate_vs_exclusive": round(sum(fr), 3)}
    print(json.dumps({"train_train_summary": summary}), flush=True)
    return out, summary


def decode_mix(small: bool = False):
    """Decode beside prefill-type work: one BERT-base-shaped inference instance
    (batches of up to 4, 200 requests/s, latency-sensitive) and one d = 2048
    decoder generating 64 tokens after a 512-token prompt for 2 sequences at a
    time, back to back (latency-sensitive: its time per output token)."""
    if small:
        inf = Served(0, "bert_inf", SMALL, 64, 4, 200.0, 0.25, 0.5, True, 51)
        gen = Generator(1, "decoder_gen", dict(SMALL, pre_ln=1, causal=1), 2, 64, 8, 0.5, 0.75, True, 56)
    else:
        inf = Served(0, "bert_inf", BERT, 128, 4, 200.0, 0.25, 0.5, True, 51)
        gen = Generator(1, "decoder_gen", DECODER, 2, 512, 64, 0.5, 0.75, True, 56)
    return [inf, gen]


def run_decode_mix(policies, horizon, warmup, period, small=False, cv=1.0, klc="device", ctl_params=None,
                   timeline=False):
    """Each policy with both instances, then each alone on the whole GPU."""
    served = decode_mix(small)
    served[0].cv, served[0].klc = cv, klc   # the inference instance's arrivals and KLC
    out, excl = run_with_exclusive(served, policies, horizon, warmup, period, ctl_params, timeline)
    summary = {}
    for r in out:
        if r["policy"].startswith("exclusive"):
            continue
        inf, gen = r["instances"]
        e_inf, e_gen = excl["bert_inf"], excl["decoder_gen"]
        summary[r.get("label", r["policy"])] = {
            "inference_p50_vs_exclusive": round(inf["p50_ms"] / e_inf["p50_ms"], 3) if inf["p50_ms"] else None,
            "inference_p95_vs_exclusive": round(inf["p95_ms"] / e_inf["p95_ms"], 3) if inf["p95_ms"] else None,
            "inference_p99_vs_exclusive": round(inf["p99_ms"] / e_inf["p99_ms"], 3) if inf["p99_ms"] else None,
            "tpot_p50_vs_exclusive": round(gen["tpot_p50_ms"] / e_gen["tpot_p50_ms"], 3) if gen["tpot_p50_ms"] else None,
            "tpot_p99_vs_exclusive": round(gen["tpot_p99_ms"] / e_gen["tpot_p99_ms"], 3) if gen["tpot_p99_ms"] else None,
            "decode_tokens_vs_exclusive": round(gen["tokens_s"] / e_gen["tokens_s"], 3) if e_gen["tokens_s"] else None}
    print(json.dumps({"decode_inf_summary": summary, "cv": cv, "klc": klc}), flush=True)
    return out, summary


def queue_probe(seconds: float = 3.0) -> list:
    """What quota switches and masked queues cost co-located instances on this
    chip: four BERT-base-shaped instances (batch 4, one host thread each, on
    disjoint 32-CU placements, two prepared each) run back-to-back batches
    while one of these happens:
      fixed    nothing (the reference);
      switch   each instance alternates between its two prepared placements
               (same size, disjoint) every batch;
      churn    a fifth instance creates a masked queue for a never-seen
               placement every 20 ms (its cache of 2 evicts one each time);
      idle+N   N more masked queues exist (idle instances' prepared masks).
    Reports each phase's per-batch device time and how many masked queues the
    process holds."""
    n_cu = ie.device_info(0)[0]
    insts = [ie.Instance(device=0, max_batch=4, max_seq=128, seed=51 + i, **BERT) for i in range(4)]
    spare = ie.Instance(device=0, max_batch=1, max_seq=128, seed=60, **BERT)
    x = torch.from_numpy(np.random.default_rng(7).standard_normal((4, 128, 768), dtype=np.float32)).to("cuda:0")
    places = [((32, 64 * i), (32, 64 * i + 32)) for i in range(len(insts))]
    for inst, (p0, p1) in zip(insts, places):
        inst.prepare_quota(*p1)
        inst.set_quota(*p0)
        inst.submit(x)
        inst.wait()
    torch.cuda.synchronize()
    rows, extra = [], []
    held = {"insts": 2 * len(insts), "spare": 0, "extra": 0}

    def phase(name, switch=False, churn=False):
        stop = threading.Event()
        times = [[] for _ in insts]

        def drive(i):
            k = 0
            while not stop.is_set():
                if switch:
                    insts[i].set_quota(*places[i][k % 2])
                insts[i].submit(x)
                insts[i].wait()
                times[i].append(insts[i].last_batch_ms())
                k += 1

        def churner():
            j = 0
            while not stop.is_set():
                spare.prepare_quota(8 + 8 * (j % 24), (8 * j) % n_cu)   # a never-seen placement each time
                j += 1
                time.sleep(0.02)

        ths = [threading.Thread(target=drive, args=(i,)) for i in range(len(insts))]
        if churn:
            ths.append(threading.Thread(target=churner))
        for t in ths:
            t.start()
        time.sleep(seconds)
        stop.set()
        for t in ths:
            t.join()
        if churn:
            held["spare"] = 2
        allt = np.concatenate([np.array(t[3:]) for t in times])
        med = float(np.median(allt))
        rows.append({"phase": name, "masked_queues": sum(held.values()), "batches": int(len(allt)),
                     "p50_ms": round(med, 3), "p99_ms": round(float(np.percentile(allt, 99)), 3),
                     "max_ms": round(float(allt.max()), 3), "over_5x_median": int((allt > 5 * med).sum())})
        print(json.dumps(rows[-1]), flush=True)

    small = dict(n_layers=1, d_model=128, n_heads=2, d_ff=512, pre_ln=0, causal=0, n_out=0)
    try:
        phase("fixed")
        phase("switch", switch=True)
        for inst, (p0, _) in zip(insts, places):
            inst.set_quota(*p0)
        phase("churn", churn=True)
        spare.close()
        held["spare"] = 0
        for n in (4, 8, 12, 16, 24):
            while 2 * len(extra) < n:
                k = len(extra)
                e = ie.Instance(device=0, max_batch=1, max_seq=32, seed=70 + k, **small)
                e.prepare_quota(8 + 8 * (k % 8), (32 * k) % n_cu)
                e.prepare_quota(16 + 8 * (k % 8), (32 * k + 8) % n_cu)
                extra.append(e)
            held["extra"] = 2 * len(extra)
            phase(f"idle+{n}")
    finally:
        for inst in insts + [spare] + extra:
            inst.close()
    return rows


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--policy", nargs="+", default=["shared", "static", "proportional", "alg2"])
    ap.add_argument("--horizon", type=float, default=20.0)
    ap.add_argument("--warmup", type=float, default=2.0)
    ap.add_argument("--period-ms", type=float, default=20.0)
    ap.add_argument("--granule", type=int, default=GRANULE, help="quota granularity (CUs) of proportional and alg2")
    ap.add_argument("--small", action="store_true", help="small models (quick functional run)")
    ap.add_argument("--mix", choices=["inference", "train", "train2", "decode"], default="inference",
                    help="inference: the four-instance serving mix; train: inference beside a training instance; "
                         "train2: two training instances; decode: inference beside a token-by-token decoder")
    ap.add_argument("--queue-probe", action="store_true",
                    help="measure what creating, switching and keeping masked queues costs co-located instances")
    ap.add_argument("--cv", type=float, default=1.0,
                    help="coefficient of variation of the inference instances' inter-arrival gaps "
                         "(1: Poisson; otherwise Gamma-distributed gaps of the same mean)")
    ap.add_argument("--klc", choices=["device", "cycle"], default="device",
                    help="KLC reported to alg2/alg2p: a batch's device time, or its cycle from the arrival of "
                         "its oldest request, each relative to the fastest batch of its size and quota")
    ap.add_argument("--eta-violation", type=float, default=None,
                    help="alg2/alg2p: relative KLC rise that raises EMERGENCY (the library's default if omitted)")
    ap.add_argument("--window", type=int, default=None,
                    help="alg2/alg2p: kernel-rate window RW in control periods (the library's default if omitted)")
    ap.add_argument("--temporary-yield", action="store_true",
                    help="alg2/alg2p: an EMERGENCY scale-down of the co-located instances leaves their plan unchanged "
                         "(IEFWD_CTL_TEMPORARY_YIELD)")
    ap.add_argument("--exclusive", action="store_true",
                    help="inference mix: also run each instance alone on the whole GPU and report latency ratios")
    ap.add_argument("--timeline", action="store_true",
                    help="add each period's quotas, controller state and arrivals to the results")
    ap.add_argument("--queue-order", choices=["rounds", "instance"], default="rounds",
                    help="order in which the paired policy prepares its placements' queues")
    args = ap.parse_args()
    ctl_params = {k: v for k, v in (("eta_violation", args.eta_violation), ("window", args.window)) if v is not None}
    if args.temporary_yield:
        ctl_params["temporary_yield"] = True
    if args.queue_probe:
        queue_probe()
        return 0
    if args.mix == "train":
        run_train_mix(args.policy, args.horizon, args.warmup, args.period_ms, args.small, args.cv, args.klc,
                      ctl_params, args.timeline)
        return 0
    if args.mix == "train2":
        run_train2_mix(args.policy, args.horizon, args.warmup, args.period_ms, args.small, ctl_params, args.timeline)
        return 0
    if args.mix == "decode":
        run_decode_mix(args.policy, args.horizon, args.warmup, args.period_ms, args.small, args.cv, args.klc,
                       ctl_params, args.timeline)
        return 0
    t = time.perf_counter()
    served = build_mix(default_mix(args.small))
    for s in served:
        s.cv, s.klc = args.cv, args.klc
    print(json.dumps({"setup_s": round(time.perf_counter() - t, 1),
                      "mix": [(s.name, s.seq, s.max_batch, s.rate, s.request, s.limit, s.slo) for s in served],
                      "cv": args.cv, "klc": args.klc}),
          flush=True)
    try:
        out = []
        for pol in args.policy:
            name, _, per = pol.partition("@")          # "alg2@100": policy with its own period in ms
            period = float(per) if per else args.period_ms
            res = run_policy(name, served, args.horizon, args.warmup, period / 1e3, args.granule, args.queue_order,
                             ctl_params, args.timeline)
            res["label"] = pol
            out.append(res)
            print(json.dumps(res), flush=True)
        if args.exclusive:
            excl = {}
            for one in served:
                res = run_policy("shared", [one], args.horizon, args.warmup, args.period_ms / 1e3)
                res["policy"] = f"exclusive:{one.name}"
                excl[one.name] = res["instances"][0]
                print(json.dumps(res), flush=True)
            summary = {}
            for r in out:
                summary[r["label"]] = {st["name"]: {f"{k}_vs_exclusive": round(st[k] / excl[st["name"]][k], 3)
                                                    for k in ("p50_ms", "p95_ms", "p99_ms")
                                                    if st[k] and excl[st["name"]][k]}
                                       for st in r["instances"]}
            print(json.dumps({"inference_summary": summary, "cv": args.cv, "klc": args.klc}), flush=True)
    finally:
        for s in served:
            s.inst.close()
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
