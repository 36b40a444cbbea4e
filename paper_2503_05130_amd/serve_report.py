"""Markdown tables from the JSON lines the serving harness prints.

  python -m paper_2503_05130_amd.serve > out.jsonl
  python -m paper_2503_05130_amd.serve_report out.jsonl      (or from stdin)

One row per (policy result, instance): the policy (its label when it ran
with its own period), the instance, its mean quota, then the figures that
apply to it: latency percentiles for request streams, steps/s for training,
TPOT for decoding, and quota switches; then each run's summary line.
"""
from __future__ import annotations

import json
import sys

STATES = {"0": "NONE", "1": "EMERGENCY", "2": "RECOVERY", "3": "CONTENTION"}


def rows(lines):
    """(header, rows) for the policy results among `lines` (decoded JSON)."""
    head = ["policy", "instance", "mean quota", "p50 ms", "p95 ms", "p99 ms", "steps/s", "TPOT p50 ms",
            "switches", "controller states"]
    out = []
    for r in lines:
        if "instances" not in r:
            continue
        label = r.get("label", r["policy"])
        quotas = r.get("mean_quota") or [None] * len(r["instances"])
        states = ", ".join(f"{STATES.get(k, k)} {v}" for k, v in r.get("state_counts", {}).items() if k != "-1")
        for q, st in zip(quotas, r["instances"]):
            cell = lambda k: "-" if st.get(k) is None else str(st[k])
            out.append([label, st["name"], "-" if q is None else str(q), cell("p50_ms"), cell("p95_ms"),
                        cell("p99_ms"), cell("steps_s"), cell("tpot_p50_ms"), cell("quota_changes"), states or "-"])
    return head, out


def markdown(head, body):
    lines = ["| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    lines += ["| " + " | ".join(r) + " |" for r in body]
    return "\n".join(lines)


def main(argv=None) -> int:
    argv = sys.argv[1:] if argv is None else argv
    text = open(argv[0]).read() if argv else sys.stdin.read()
    lines = [json.loads(x) for x in text.splitlines() if x.startswith("{")]
    print(markdown(*rows(lines)))
    for r in lines:
        for key in r:
            if key.endswith("_summary"):
                print()
                print(f"{key}: {json.dumps(r[key])}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
