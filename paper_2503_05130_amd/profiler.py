"""Inference profiling on one GPU: the paper's Hybrid Growth Search Strategy
(HGSS, Sec. 3.2 "Inference Profiling") over <IBS, SMR>, with CU quotas as
the SM rate, against a full traversal of the same grid (the comparison of
Table "tab:mp-compar").

  python -m paper_2503_05130_amd.profiler [--slo-ms 100] [--models bert decoder] [--train]

What the paper fixes:
  * throughput efficacy TE = IBS / (t_exec * SMR), with the execution budget
    t_exec = SLO / 2 (a configuration is feasible when its batch time is at
    most SLO / 2);
  * the search doubles IBS at every step and raises SMR linearly by a fixed
    step (10 units), and stops at the first SLO violation (its GPT2-large
    example path: <1, 10>, <2, 20>, <4, 30>, <8, 40> violates, stop);
  * request = the SMR of the most cost-efficient feasible setting (max TE),
    limit = 2 x request.

Readings where it is silent: the SMR unit is percent of the device, realised
as the XCD-balanced CU quota round(SMR% * n_cu / n_xcd) * n_xcd; if the very
first setting violates, SMR keeps climbing at that IBS until one is feasible
(otherwise heavy models could never be placed); IBS is capped by the
instance's batch capacity and SMR at 100%; the limit is capped at 100%.

Training profiling (the same section) is a binary search over the SM rate
for the request (p = 80% of the full-GPU throughput) and limit (p = 100%)
quotas: train_binary_search, against train_traversal of every quota.

Two walks are provided.  "diagonal" is the printed path: both coordinates
grow every step.  It ties SMR to IBS, so it cannot reach large batches at a
small SM rate, where TE is usually highest.  "frontier" is a variant of the
same growth rules: IBS doubles while the setting is feasible and SMR grows by
the step only on a violation, so it visits the smallest feasible SMR of every
IBS (the settings where TE is highest at each IBS, when time falls with SMR
and grows with IBS) and stops when even 100% violates.
"""
from __future__ import annotations

import argparse
import json
import time
from typing import Callable

import numpy as np


def smr_to_cus(smr_pct: float, n_cu: int = 256, n_xcd: int = 8) -> int:
    """SM rate in percent -> XCD-balanced CU quota (at least one CU per XCD)."""
    return int(max(n_xcd, min(n_cu, round(smr_pct / 100.0 * n_cu / n_xcd) * n_xcd)))


def throughput_efficacy(ibs: int, t_ms: float, smr_pct: float) -> float:
    """TE = IBS / (t_exec * SMR): sequences per second per percent of the device."""
    return ibs / (t_ms * 1e-3 * smr_pct)


def hgss(measure: Callable[[int, float], float], slo_ms: float, ibs0: int = 1, smr0: float = 10.0,
         smr_step: float = 10.0, max_ibs: int = 256, walk: str = "diagonal") -> dict:
    """Hybrid growth search.  measure(ibs, smr_pct) -> batch time in ms."""
    if walk not in ("diagonal", "frontier"):
        raise ValueError("walk must be 'diagonal' or 'frontier'")
    budget = slo_ms / 2.0
    trials, ibs, smr = [], ibs0, smr0
    while True:
        t = measure(ibs, smr)
        ok = t <= budget
        trials.append({"ibs": ibs, "smr": smr, "t_ms": t, "feasible": ok,
                       "te": throughput_efficacy(ibs, t, smr) if ok else None})
        feasible_seen = any(tr["feasible"] for tr in trials)
        if not ok:
            if smr >= 100.0 or (walk == "diagonal" and feasible_seen):
                break                            # diagonal: first violation after a feasible setting
            smr = min(100.0, smr + smr_step)     # more SMR at this IBS
            continue
        if ibs * 2 > max_ibs:
            break
        if walk == "diagonal":
            if smr >= 100.0:
                break
            ibs, smr = ibs * 2, min(100.0, smr + smr_step)
        else:
            ibs = ibs * 2
    return _result(trials)


def traversal(measure: Callable[[int, float], float], slo_ms: float, ibs_list, smr_list) -> dict:
    """Every <IBS, SMR> of the grid."""
    budget = slo_ms / 2.0
    trials = []
    for ibs in ibs_list:
        for smr in smr_list:
            t = measure(ibs, smr)
            ok = t <= budget
            trials.append({"ibs": ibs, "smr": smr, "t_ms": t, "feasible": ok,
                           "te": throughput_efficacy(ibs, t, smr) if ok else None})
    return _result(trials)


def _result(trials) -> dict:
    feas = [t for t in trials if t["feasible"]]
    best = max(feas, key=lambda t: t["te"]) if feas else None
    out = {"trials": len(trials), "path": [(t["ibs"], t["smr"]) for t in trials], "best": best}
    if best:
        out["request_smr"] = best["smr"]
        out["limit_smr"] = min(100.0, 2 * best["smr"])
        out["ibs"] = best["ibs"]
    return out


def train_binary_search(measure: Callable[[int], float], p: float, n_cu: int = 256, n_xcd: int = 8,
                        band: float = 0.02, tight: bool = False) -> dict:
    """Training profiling (Sec. 3.2): the SM rate at which a training
    function's throughput reaches p of its full-GPU throughput T1.

    measure(quota_cus) -> throughput.  T1 at high = 100%; then mid = (low +
    high) / 2 with low = 0: below T1 p -> low = mid, else high = mid, until
    the throughput is within T1 p +- band T1.  Readings: the band is a
    fraction of T1; SMR maps to XCD-balanced CU quotas, so the search also
    ends when low and high give adjacent quotas, with high's SMR as the result
    (the smallest measured setting not below the band).

    The printed rule stops at the first setting inside the band, which need
    not be the smallest one (a throughput that saturates early is inside the
    band at 50%).  tight=True keeps bisecting below a setting inside the band
    (high = mid) until low and high are adjacent, and returns the smallest
    setting found inside or above the band."""
    trials = []

    def run(smr):
        q = smr_to_cus(smr, n_cu, n_xcd)
        t = measure(q)
        trials.append({"smr": smr, "quota_cus": q, "throughput": t})
        return t

    t1 = run(100.0)
    target, tol = p * t1, band * t1
    low, high, found = 0.0, 100.0, None
    while True:
        mid = (low + high) / 2.0
        t = run(mid)
        if abs(t - target) <= tol and not tight:
            found = mid
            break
        if t < target - tol or (not tight and t < target):
            low = mid
        else:
            high = mid
        if smr_to_cus(high, n_cu, n_xcd) - smr_to_cus(low, n_cu, n_xcd) <= n_xcd:
            found = high
            break
    return {"p": p, "smr": found, "quota_cus": smr_to_cus(found, n_cu, n_xcd), "t1": t1, "trials": len(trials),
            "path": [(tr["smr"], tr["quota_cus"]) for tr in trials]}


def train_traversal(measure: Callable[[int], float], p: float, n_cu: int = 256, n_xcd: int = 8,
                    band: float = 0.02) -> dict:
    """Every XCD-balanced quota: the smallest whose throughput is at least
    (p - band) of the full-GPU throughput."""
    quotas = list(range(n_xcd, n_cu + 1, n_xcd))
    tput = {q: measure(q) for q in quotas}
    t1 = tput[n_cu]
    ok = [q for q in quotas if tput[q] >= (p - band) * t1]
    return {"p": p, "quota_cus": min(ok), "t1": t1, "trials": len(quotas)}


class TrainTimer:
    """measure(quota) for a training instance: sequences per second from the
    median device time of a few steps at that quota."""

    def __init__(self, shape: dict, seq: int, batch: int, seed: int, n_warm: int = 1, n_time: int = 3):
        import torch

        import paper_2503_05130_amd as ie
        self.ie = ie
        self.tr = ie.Trainer(device=0, max_batch=batch, max_seq=seq, seed=seed, **shape)
        rng = np.random.default_rng(seed)
        self.x = torch.from_numpy(rng.standard_normal((batch, seq, shape["d_model"]), dtype=np.float32)).to("cuda:0")
        self.labels = torch.from_numpy(rng.integers(0, shape["n_out"], size=(batch, seq), dtype=np.int32)).to("cuda:0")
        self.batch, self.n_warm, self.n_time = batch, n_warm, n_time
        self.cache = {}

    def __call__(self, quota: int) -> float:
        if quota not in self.cache:
            self.tr.set_quota(quota)
            ms = []
            for k in range(self.n_warm + self.n_time):
                self.tr.step(self.x, self.labels)
                self.tr.wait()
                if k >= self.n_warm:
                    ms.append(self.tr.last_batch_ms())
            self.cache[quota] = self.batch / (float(np.median(ms)) * 1e-3)
        return self.cache[quota]

    def close(self):
        self.tr.close()


def profile_training(name, shape, seq, batch, seed):
    """Request (p = 80%) and limit (p = 100%) quotas by binary search, against
    a traversal of every XCD-balanced quota."""
    timer = TrainTimer(shape, seq, batch, seed)
    try:
        out = {"model": name, "seq": seq, "batch": batch}
        for p, key in ((0.8, "request"), (1.0, "limit")):
            for tight in (False, True):
                t0 = time.perf_counter()
                bs = train_binary_search(timer, p, tight=tight)
                out[key + ("_tight" if tight else "")] = dict(bs, seconds=round(time.perf_counter() - t0, 2))
        t0 = time.perf_counter()
        for p, key in ((0.8, "request_traversal"), (1.0, "limit_traversal")):
            out[key] = train_traversal(timer, p)
        out["traversal_seconds"] = round(time.perf_counter() - t0, 2)
        out["throughput_by_quota"] = {q: round(v, 1) for q, v in sorted(timer.cache.items())}
    finally:
        timer.close()
    return out


# ------------------------------------------------------------------ measuring real instances
BERT = dict(n_layers=12, d_model=768, n_heads=12, d_ff=3072, pre_ln=0, causal=0, n_out=2)
DECODER = dict(n_layers=24, d_model=2048, n_heads=16, d_ff=8192, pre_ln=1, causal=1, n_out=2)


class InstanceTimer:
    """measure(ibs, smr) for one model: median device time of a few batches."""

    def __init__(self, shape: dict, seq: int, max_ibs: int, seed: int, n_warm: int = 2, n_time: int = 5):
        import torch

        import paper_2503_05130_amd as ie
        self.ie = ie
        self.n_cu, self.n_xcd = ie.device_info(0)
        self.inst = ie.Instance(device=0, max_batch=max_ibs, max_seq=seq, seed=seed, **shape)
        rng = np.random.default_rng(seed)
        self.x = torch.from_numpy(rng.standard_normal((max_ibs, seq, shape["d_model"]), dtype=np.float32)).to("cuda:0")
        self.n_warm, self.n_time = n_warm, n_time
        self.cache = {}

    def __call__(self, ibs: int, smr: float) -> float:
        key = (ibs, smr)
        if key not in self.cache:
            self.inst.set_quota(smr_to_cus(smr, self.n_cu, self.n_xcd))
            xs = self.x[:ibs]
            times = []
            for k in range(self.n_warm + self.n_time):
                self.inst.submit(xs)
                self.inst.wait()
                if k >= self.n_warm:
                    times.append(self.inst.last_batch_ms())
            self.cache[key] = float(np.median(times))
        return self.cache[key]

    def close(self):
        self.inst.close()


def profile_model(name, shape, seq, max_ibs, slo_ms, seed):
    timer = InstanceTimer(shape, seq, max_ibs, seed)
    try:
        t0 = time.perf_counter()
        h = hgss(timer, slo_ms, max_ibs=max_ibs)
        t_h = time.perf_counter() - t0
        timer.cache.clear()
        f = hgss(timer, slo_ms, max_ibs=max_ibs, walk="frontier")
        timer.cache.clear()
        ibs_list = [1 << k for k in range(int(np.log2(max_ibs)) + 1)]
        smr_list = [10.0 * k for k in range(1, 11)]
        t0 = time.perf_counter()
        tr = traversal(timer, slo_ms, ibs_list, smr_list)
        t_t = time.perf_counter() - t0
    finally:
        timer.close()
    def ratio(r):
        return round(r["best"]["te"] / tr["best"]["te"], 4) if r.get("best") and tr.get("best") else None

    return {"model": name, "seq": seq, "slo_ms": slo_ms,
            "hgss": {k: h.get(k) for k in ("trials", "path", "request_smr", "limit_smr", "ibs")},
            "hgss_best": h.get("best"), "hgss_s": round(t_h, 2),
            "frontier": {k: f.get(k) for k in ("trials", "path", "request_smr", "limit_smr", "ibs")},
            "frontier_best": f.get("best"), "te_frontier_over_traversal": ratio(f),
            "traversal": {k: tr.get(k) for k in ("trials", "request_smr", "limit_smr", "ibs")},
            "traversal_best": tr.get("best"), "traversal_s": round(t_t, 2),
            "te_hgss_over_traversal": ratio(h)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--slo-ms", type=float, default=100.0)
    ap.add_argument("--models", nargs="+", default=["bert", "decoder"])
    ap.add_argument("--train", action="store_true",
                    help="training profiling of the BERT-base-shaped encoder (batch 32 x 128) instead")
    args = ap.parse_args()
    if args.train:
        print(json.dumps(profile_training("bert_base_l12_d768_s128 training", BERT, 128, 32, 65)), flush=True)
        return 0
    specs = {"bert": ("bert_base_l12_d768_s128", BERT, 128, 256, 61),
             "decoder": ("decoder_l24_d2048_s1024", DECODER, 1024, 8, 63)}
    for m in args.models:
        name, shape, seq, max_ibs, seed = specs[m]
        print(json.dumps(profile_model(name, shape, seq, max_ibs, args.slo_ms, seed)), flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
