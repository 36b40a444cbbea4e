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
  R2  "scaled down by the KLC change": Alg. 2 divides by dT, which for
      dT < 1 would scale the instance *up*; we divide by the KLC ratio
      1 + dT = T_current / T_min of the instance that raised EMERGENCY.
  R3  the SLO scale-up branch is uncapped in Alg. 2; tokens here are CUs,
      so it is capped at MaxTokens.
  R4  SLO-sensitive instances are evaluated first in a period (they set the
      shared state), then the others, each group in id order.
  R5  T_current is the KLC reported for the current period, T_min the
      smallest ever reported.  A period in which the instance completed no
      iteration has no T_current and its dT is 0: nothing was seen to slow
      down.  (Holding the previous period's KLC instead would keep an instance
      that went idle after a violation in EMERGENCY, so the text's rule that
      an instance with no recent kernels scales down could never follow an
      EMERGENCY.)  Before any KLC is reported dT = 0.  R_last starts at
      MaxTokens * request.  RW holds the last `window` kernel counts.
  R6  tokens become a CU quota: round(R / granule) * granule, clamped to
      [min_quota, MaxTokens].  A CU mask cannot be oversubscribed without the
      instances slowing each other down (and with a batch in flight on its old
      mask, an instance moved onto those CUs waits behind it), so placements
      never overlap: the SLO-sensitive quotas are shrunk until every other
      instance can keep min_quota, then the others are shrunk into the CUs that
      remain; shrinking keeps min_quota each and shares the rest in proportion
      to each quota's excess over min_quota (rounded down to the granule).  SLO-sensitive
      instances take mask bits upward from 0 (id order), the others downward
      from the top (id order), so a change of one quota moves one boundary.

  R8  the text calls the co-located instances' scale-down under EMERGENCY
      temporary, while Alg. 2 keeps R_last in CONTENTION, so that a
      scale-down is undone only through RECOVERY (the SLO instance idle for a
      whole window).  Both are offered: by default (temporary_yield False) a
      yielded issue becomes R_last, as Alg. 2 reads; with temporary_yield
      True a yielded issue does not replace R_last, so the yield is computed
      from the plan held before the emergency (consecutive EMERGENCY periods
      do not compound it) and CONTENTION afterwards restores that plan.

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
    t_current: float = 0.0          # 0: no KLC this period
    t_min: float = math.inf
    dt: float = 0.0


class Controller:
    """IssueToken (Alg. 2) for a set of co-located instances."""

    def __init__(self, max_tokens=256, window=4, granule=8, min_quota=8, eta_violation=0.2, eta_increase=1.25,
                 temporary_yield=False):
        self.max_tokens = float(max_tokens)
        self.n_cu = int(max_tokens)
        self.window = int(window)
        self.granule = int(granule)
        self.min_quota = int(min_quota)
        self.eta_violation = float(eta_violation)
        self.eta_increase = float(eta_increase)
        self.temporary_yield = bool(temporary_yield)
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
        inst.dt = (inst.t_current - inst.t_min) / inst.t_min if inst.t_current > 0 else 0.0
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
        yielded = self.state == EMERGENCY and self.temporary_yield
        for i, inst in enumerate(self.insts):
            if inst.slo or not yielded:        # a temporary yield leaves the plan R_last as it was
                inst.r_last = out[i]
            inst.r_current = 0
            inst.t_current = 0.0           # the next period starts with no KLC
        return out

    def _fit(self, qs, idx, avail):
        """Shrink the quotas qs[i], i in idx, to sum to at most avail: each keeps
        min_quota and the rest of avail is shared in proportion to its excess
        over min_quota, rounded down to the granule."""
        want = sum(qs[i] for i in idx)
        if not idx or want <= avail:
            return
        spare = max(avail - len(idx) * self.min_quota, 0)
        excess = want - len(idx) * self.min_quota
        for i in idx:
            extra = ((qs[i] - self.min_quota) * spare // excess) // self.granule * self.granule if excess else 0
            qs[i] = self.min_quota + extra

    def quotas(self, tokens: list[float]) -> tuple[list[int], list[int]]:
        """Tokens -> (CU quota, first mask bit) per instance (reading R6)."""
        n = len(tokens)
        qs = []
        for r in tokens:
            q = int(math.floor(r / self.granule + 0.5)) * self.granule
            qs.append(max(self.min_quota, min(self.n_cu, q)))
        slo = [i for i in range(n) if self.insts[i].slo]
        other = [i for i in range(n) if not self.insts[i].slo]
        self._fit(qs, slo, self.n_cu - len(other) * self.min_quota)
        self._fit(qs, other, self.n_cu - sum(qs[i] for i in slo))
        firsts = [0] * n
        lo, hi = 0, self.n_cu
        for i in slo:
            firsts[i] = lo % self.n_cu
            lo += qs[i]
        for i in other:
            hi -= qs[i]
            firsts[i] = hi % self.n_cu
        return qs, firsts
