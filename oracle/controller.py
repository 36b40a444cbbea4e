"""Oracle for the quota controller: the paper's fast scale-up/down control
(Sec. 3.4.1, Alg. 2, "IssueToken"), written out plainly in fp64.

Test infrastructure only (see oracle/__init__.py): nothing in the product
imports it.

What the paper fixes (Sec. 3.4.1 and Alg. 2):
  * every control period each co-located instance gets an issue R_issue of
    tokens; inputs are MaxTokens, a sliding window RW of each instance's recent
    kernel rates, the instance's <request, limit> (fractions of MaxTokens), its
    type (SLO-sensitive or not) and its current / minimum kernel launching
    cycle (KLC, the duration of one iteration -- for inference one batch);
  * SLO-sensitive instances: dT = (T_current - T_min) / T_min;
      dT > eta_violation          -> EMERGENCY,  MaxTokens * limit
      its own window all zero     -> RECOVERY,   MaxTokens * request (scale down)
      every other window all zero -> RECOVERY,   R_last * eta_increase (scale up)
      otherwise                   -> CONTENTION, MaxTokens * request;
  * other instances act on the shared state:
      NONE (no co-located SLO instance) -> MaxTokens * limit
      EMERGENCY  -> min(MaxTokens * request, R_last) scaled down by the KLC change
      RECOVERY   -> min(R_last * eta_increase, MaxTokens * limit)
      CONTENTION -> R_last;
  * only the instance that raised EMERGENCY can reset or change it.

Readings where the paper is silent or ambiguous (each also listed in the
design notes):
  R1  eta_violation and eta_increase are not given: defaults 0.2 and 1.25.
  R2  "scaled down by the KLC change": the listing divides by dT, which for
      dT < 1 would scale the instance *up*; we divide by the KLC ratio
      1 + dT = T_current / T_min of the instance that raised EMERGENCY.
  R3  the SLO scale-up branch is uncapped in the listing; tokens here are CUs,
      so it is capped at MaxTokens.
  R4  SLO-sensitive instances are evaluated first in a period (they set the
      shared state), then the others, each group in id order.
  R5  T_current is the most recent reported KLC, T_min the smallest ever
      reported; before any KLC is reported dT = 0.  R_last starts at
      MaxTokens * request.  RW holds the last `window` kernel counts.
  R6  tokens become a CU quota: round(R / granule) * granule, clamped to
      [min_quota, MaxTokens]; instances are placed on consecutive mask bits in
      id order (first_0 = 0, first_i = first_{i-1} + quota_{i-1} mod n_cu).

Parity unpinned against numbers printed in the paper (it prints no controller
traces); pinned against the behaviour its text describes (tests).
"""
from __future__ import annotations

import math
from collections import deque
from dataclasses import dataclass, field

NONE, EMERGENCY, RECOVERY, CONTENTION = 0, 1, 2, 3


@dataclass
class _Inst:
    request: float
    limit: float
    slo: bool
    window: int
    rw: deque = field(default_factory=deque)
    r_last: float = 0.0
    r_current: int = 0
    t_current: float = 0.0
    t_min: float = math.inf
    dt: float = 0.0


class Controller:
    """IssueToken (Alg. 2) for a set of co-located instances."""

    def __init__(self, max_tokens=256, window=4, granule=8, min_quota=8, eta_violation=0.2, eta_increase=1.25):
        self.max_tokens = float(max_tokens)
        self.n_cu = int(max_tokens)
        self.window = int(window)
        self.granule = int(granule)
        self.min_quota = int(min_quota)
        self.eta_violation = float(eta_violation)
        self.eta_increase = float(eta_increase)
        self.insts: list[_Inst] = []
        self.state = NONE
        self.owner = -1            # instance that raised EMERGENCY
        self.owner_dt = 0.0

    def add(self, request: float, limit: float, slo_sensitive: bool) -> int:
        inst = _Inst(float(request), float(limit), bool(slo_sensitive), self.window)
        inst.r_last = self.max_tokens * inst.request
        self.insts.append(inst)
        return len(self.insts) - 1

    def report(self, i: int, kernels: int, klc_ms: float) -> None:
        """Kernels launched by instance i during the period, and the KLC of its
        last completed iteration (<= 0: none completed in this period)."""
        inst = self.insts[i]
        inst.r_current = int(kernels)
        if klc_ms > 0:
            inst.t_current = float(klc_ms)
            inst.t_min = min(inst.t_min, float(klc_ms))

    def _issue_slo(self, i: int) -> float:
        inst = self.insts[i]
        inst.dt = (inst.t_current - inst.t_min) / inst.t_min if inst.t_min < math.inf else 0.0
        others_idle = all(sum(o.rw) == 0 for j, o in enumerate(self.insts) if j != i)
        if inst.dt > self.eta_violation:
            state, r = EMERGENCY, self.max_tokens * inst.limit
        elif sum(inst.rw) == 0:
            state, r = RECOVERY, self.max_tokens * inst.request
        elif others_idle:
            state, r = RECOVERY, min(inst.r_last * self.eta_increase, self.max_tokens)
        else:
            state, r = CONTENTION, self.max_tokens * inst.request
        # only the instance that raised EMERGENCY may change it
        if self.state != EMERGENCY or self.owner == i:
            self.state = state
            self.owner = i if state == EMERGENCY else -1
            self.owner_dt = inst.dt if state == EMERGENCY else 0.0
        return r

    def _issue_other(self, i: int) -> float:
        inst = self.insts[i]
        if self.state == NONE:
            return self.max_tokens * inst.limit
        if self.state == EMERGENCY:
            return min(self.max_tokens * inst.request, inst.r_last) / (1.0 + self.owner_dt)
        if self.state == RECOVERY:
            return min(inst.r_last * self.eta_increase, self.max_tokens * inst.limit)
        return inst.r_last

    def issue(self) -> list[float]:
        """One control period: R_issue for every instance, in id order."""
        for inst in self.insts:
            inst.rw.append(inst.r_current)
            while len(inst.rw) > self.window:
                inst.rw.popleft()
        if not any(inst.slo for inst in self.insts):
            self.state, self.owner, self.owner_dt = NONE, -1, 0.0
        out = [0.0] * len(self.insts)
        for i, inst in enumerate(self.insts):
            if inst.slo:
                out[i] = self._issue_slo(i)
        for i, inst in enumerate(self.insts):
            if not inst.slo:
                out[i] = self._issue_other(i)
        for i, inst in enumerate(self.insts):
            inst.r_last = out[i]
            inst.r_current = 0
        return out

    def quotas(self, tokens: list[float]) -> tuple[list[int], list[int]]:
        """Tokens -> (CU quota, first mask bit) per instance (reading R6)."""
        qs, firsts, first = [], [], 0
        for r in tokens:
            q = int(math.floor(r / self.granule + 0.5)) * self.granule
            q = max(self.min_quota, min(self.n_cu, q))
            qs.append(q)
            firsts.append(first)
            first = (first + q) % self.n_cu
        return qs, firsts
