"""Co-located serving with a quota policy per control period (small models,
short horizon): every request is served under each policy and the controller
re-masks the instances; also under bursty (Gamma) arrivals with the cycle KLC."""
import numpy as np
import pytest

from paper_2503_05130_amd import serve

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def served():
    s = serve.build_mix(serve.default_mix(small=True))
    yield s
    for x in s:
        x.inst.close()


@pytest.mark.parametrize("policy", ["shared", "static", "proportional", "alg2", "paired", "alg2p"])
def test_policy_serves_every_request(served, policy):
    print(f"serve policy={policy}", flush=True)
    res = serve.run_policy(policy, served, horizon=1.5, warmup=0.2, period=0.01)
    print(res, flush=True)
    for st in res["instances"]:
        assert st["dropped"] == 0, st
        assert st["requests"] > 0 and st["p99_ms"] is not None and st["p99_ms"] >= st["p50_ms"] > 0
    assert res["periods"] > 10
    q = np.array(res["mean_quota"])
    assert np.all((q >= 8) & (q <= 256))
    if policy in ("alg2", "alg2p"):
        assert sum(res["state_counts"].values()) == res["periods"]
    if policy in ("paired", "alg2p"):
        # quotas from the fixed vocabulary only: each instance uses at most the 3 placements of its pair
        for st in res["instances"]:
            assert st["distinct_placements"] <= 3, st
        assert np.all((q >= 32) & (q <= 96))        # means of quotas in {32, 64, 96}
    agg = res["aggregate"]
    assert agg["requests_s"] > 0 and agg["p99_ms"] >= agg["p50_ms"] > 0


def test_training_beside_inference():
    """The train-inf mix (small models): the inference instance serves every
    request and the training instance completes steps under each policy, and
    both also alone."""
    out, summary = serve.run_train_mix(["static", "alg2"], horizon=1.5, warmup=0.2, period=10.0, small=True)
    names = [r["policy"] for r in out]
    assert names == ["static", "alg2", "exclusive:bert_inf", "exclusive:bert_train"]
    for r in out:
        for st in r["instances"]:
            if st.get("training"):
                assert st["steps"] > 0 and st["steps_s"] > 0
            else:
                assert st["dropped"] == 0 and st["requests"] > 0
    for pol in ("static", "alg2"):
        v = summary[pol]
        assert v["inference_p50_vs_exclusive"] > 0 and v["training_throughput_vs_exclusive"] > 0


def test_decode_beside_inference():
    """The decode mix (small models): the inference instance serves every
    request and the decoder completes decode steps under each policy, and both
    also alone."""
    out, summary = serve.run_decode_mix(["static", "alg2"], horizon=1.5, warmup=0.2, period=10.0, small=True)
    names = [r["policy"] for r in out]
    assert names == ["static", "alg2", "exclusive:bert_inf", "exclusive:decoder_gen"]
    for r in out:
        for st in r["instances"]:
            if st.get("decoding"):
                assert st["steps"] > 0 and st["tokens_s"] > 0 and st["tpot_p99_ms"] >= st["tpot_p50_ms"] > 0
            else:
                assert st["dropped"] == 0 and st["requests"] > 0
    for pol in ("static", "alg2"):
        v = summary[pol]
        assert v["inference_p50_vs_exclusive"] > 0 and v["tpot_p50_vs_exclusive"] > 0


@pytest.mark.parametrize("temporary_yield", [False, True])
def test_training_beside_bursty_inference(temporary_yield):
    """Gamma arrivals at CV 4 into the inference instance, the cycle KLC, and
    either yield reading of the controller (small models): every request is
    served, training completes steps, and the controller's parameters are
    recorded with the result."""
    params = {"temporary_yield": True} if temporary_yield else None
    print(f"train mix cv 4 klc cycle temporary_yield={temporary_yield}", flush=True)
    out, summary = serve.run_train_mix(["alg2"], horizon=1.5, warmup=0.2, period=10.0, small=True, cv=4.0,
                                       klc="cycle", ctl_params=params, timeline=True)
    alg2 = out[0]
    assert alg2["policy"] == "alg2" and alg2.get("ctl_params") == params
    # the timeline: one entry per period, quotas within the device, the requests
    # of the inference instance counted once each
    tl = alg2["timeline"]
    assert len(tl) == alg2["periods"]
    assert all(len(q) == 2 and all(32 <= x <= 256 for x in q) and st in (1, 2, 3) for _, q, st, _ in tl)
    assert [t for t, _, _, _ in tl] == sorted(t for t, _, _, _ in tl)
    arrived = sum(a[0] for _, _, _, a in tl)
    assert arrived > 0
    assert all(a[1] is None for _, _, _, a in tl)      # the training instance has no arrivals
    assert sum(alg2["state_counts"].values()) == alg2["periods"] > 10
    inf, trn = alg2["instances"]
    assert inf["dropped"] == 0 and inf["requests"] > 0
    assert inf["p99_ms"] >= inf["p95_ms"] >= inf["p50_ms"] > 0
    assert inf["klc_ratio_p50_p90"] is not None and inf["klc_ratio_p50_p90"][0] >= 0.99
    assert trn["steps"] > 0
    assert summary["alg2"]["inference_p95_vs_exclusive"] > 0


def test_paired_policies_beside_training():
    """One pair (inference beside training, small models) owns the whole
    device: the paired and alg2p policies move its split among quarters of
    the 256 CUs, every request is served and training completes steps."""
    print("train mix paired alg2p", flush=True)
    out, summary = serve.run_train_mix(["paired", "alg2p"], horizon=1.5, warmup=0.2, period=10.0, small=True)
    assert [r["policy"] for r in out][:2] == ["paired", "alg2p"]
    for r in out[:2]:
        inf, trn = r["instances"]
        assert inf["dropped"] == 0 and inf["requests"] > 0 and trn["steps"] > 0
        for st in (inf, trn):
            assert st["distinct_placements"] <= 3, st
        q = np.array(r["mean_quota"])
        # a grow is issued only once the partner has left the CUs, so the
        # two quotas of a period sum to at most the device
        assert np.all((q >= 64) & (q <= 192)) and q.sum() <= 256 + 1e-6, q


def test_training_beside_training():
    """The train-train mix (small models): both training instances complete
    steps under each policy and alone, and the aggregate of their normalised
    throughputs is reported."""
    print("train2 mix", flush=True)
    out, summary = serve.run_train2_mix(["static", "alg2"], horizon=1.5, warmup=0.2, period=10.0, small=True)
    assert [r["policy"] for r in out] == ["static", "alg2", "exclusive:train_a", "exclusive:train_b"]
    for r in out:
        for st in r["instances"]:
            assert st["training"] and st["steps"] > 0
    for pol in ("static", "alg2"):
        v = summary[pol]
        assert len(v["throughput_vs_exclusive"]) == 2 and v["aggregate_vs_exclusive"] > 0
    # no SLO-sensitive instance: the controller stays in NONE and splits the CUs
    assert out[1]["state_counts"] == {"0": out[1]["periods"]}


def test_paired_policies_beside_decoding():
    """The decode mix (small models) under the paired policies: its two
    instances form one pair over the whole device; every request is served and
    the decoder completes decode steps."""
    print("decode mix paired alg2p", flush=True)
    out, summary = serve.run_decode_mix(["paired", "alg2p"], horizon=1.5, warmup=0.2, period=10.0, small=True)
    for r in out[:2]:
        inf, gen = r["instances"]
        assert inf["dropped"] == 0 and inf["requests"] > 0 and gen["steps"] > 0
        for st in (inf, gen):
            assert st["distinct_placements"] <= 3, st
        q = np.array(r["mean_quota"])
        assert np.all((q >= 64) & (q <= 192)) and q.sum() <= 256 + 1e-6, q


def test_inference_mix_cli_with_exclusive(monkeypatch, capsys):
    """The command line on the four-instance mix (small models): a policy,
    then every instance alone, and the latency ratios against exclusive."""
    import json
    import sys
    print("cli inference mix --exclusive", flush=True)
    monkeypatch.setattr(sys, "argv", ["serve", "--small", "--policy", "static", "--horizon", "1.5", "--warmup", "0.2",
                                      "--cv", "2", "--klc", "cycle", "--exclusive"])
    assert serve.main() == 0
    lines = [json.loads(x) for x in capsys.readouterr().out.splitlines() if x.startswith("{")]
    names = [x.get("policy") for x in lines if "policy" in x]
    assert names == ["static", "exclusive:enc_a", "exclusive:enc_b", "exclusive:dec_a", "exclusive:dec_b"]
    summary = lines[-1]["inference_summary"]["static"]
    assert set(summary) == {"enc_a", "enc_b", "dec_a", "dec_b"}
    assert all(v["p95_ms_vs_exclusive"] > 0 for v in summary.values())
