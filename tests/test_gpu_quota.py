"""Quota layer on the GPU: a CU-masked stream confines an instance's
workgroups to the CUs of its mask, spread evenly over the XCDs."""
import collections

import numpy as np
import pytest
import torch

import paper_2503_05130_amd as ie
import workloads as W
from tests.gpu_util import DEV, instance_config, run_instance

pytestmark = pytest.mark.gpu


def probe(stream_handle, n_groups=8192):
    out = torch.zeros(2 * n_groups, dtype=torch.int32, device=DEV)
    ie.test_cu_probe(n_groups, out, stream=stream_handle)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.uint32).reshape(-1, 2)


def observed_cus(stream_handle, n_groups=8192):
    v = probe(stream_handle, n_groups)
    xcc = v[:, 0] & 0xF
    cu = (v[:, 1] >> 8) & 0xFF          # CU, shader-array and shader-engine fields of HW_ID
    return set(zip(xcc.tolist(), cu.tolist()))


def test_device_info():
    n_cu, n_xcd = ie.device_info(0)
    print(f"device: {n_cu} CUs, {n_xcd} XCDs", flush=True)
    assert n_cu == 256 and n_xcd == 8


@pytest.mark.parametrize("q", [8, 24, 64, 128, 192, 256])
def test_masked_stream_residency(q):
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    with ie.Instance(**instance_config(shape, 1, 32)) as inst:
        inst.set_quota(q)
        run_instance(inst, W.make_input(1, 1, 32, 128))     # applies the mask
        cus = observed_cus(inst.stream_handle())
    per_xcc = collections.Counter(x for x, _ in cus)
    print(f"quota {q}: {len(cus)} CUs seen, per XCC {sorted(per_xcc.items())}", flush=True)
    assert len(cus) == q
    assert len(per_xcc) == min(8, q)
    assert max(per_xcc.values()) - min(per_xcc.values()) <= 1


@pytest.mark.parametrize("q,first", [(64, 64), (128, 128), (24, 250)])
def test_placed_stream_residency(q, first):
    # a quota placed at `first` runs on exactly the CUs of its mask: two
    # placements that do not overlap in the mask see disjoint CU sets
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    with ie.Instance(**instance_config(shape, 1, 32)) as a, ie.Instance(**instance_config(shape, 1, 32)) as b:
        a.set_quota(q, first)
        b.set_quota(q, (first + q) % 256)
        x = W.make_input(1, 1, 32, 128)
        run_instance(a, x)
        run_instance(b, x)
        ca, cb = observed_cus(a.stream_handle()), observed_cus(b.stream_handle())
    print(f"quota {q} at {first}: {len(ca)} and {len(cb)} CUs, overlap {len(ca & cb)}", flush=True)
    assert len(ca) == q and len(cb) == q
    assert not (ca & cb)


def test_prepare_from_another_thread():
    # a controller thread prepares masked streams while the instance serves;
    # switching to a prepared quota is then cheap and lands on the right CUs
    import threading
    import time
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    x = W.make_input(1, 1, 32, 128)
    with ie.Instance(**instance_config(shape, 1, 32)) as inst:
        run_instance(inst, x)
        plans = [(32 * (i + 1), (32 * i) % 256) for i in range(6)]
        errors = []

        def prep():
            try:
                for q, f in plans:
                    inst.prepare_quota(q, f)
            except Exception as e:        # surfaced below
                errors.append(e)

        t = threading.Thread(target=prep)
        t.start()
        for _ in range(20):
            run_instance(inst, x)
        t.join(timeout=60)
        assert not errors, errors
        for q, f in plans[-4:]:
            inst.set_quota(q, f)
            t0 = time.perf_counter()
            run_instance(inst, x)
            ms = (time.perf_counter() - t0) * 1e3
            cus = observed_cus(inst.stream_handle())
            print(f"prepared quota {q} at {f}: first batch {ms:.2f} ms, {len(cus)} CUs", flush=True)
            assert len(cus) == q


def test_stream_cache_capacity():
    # a cache sized for a fixed set of placements: switching among them gives the
    # same bits and the right masks; shrinking it keeps the stream in use
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    x = W.make_input(7, 2, 32, 128)
    with ie.Instance(**instance_config(shape, 2, 32)) as inst:
        ref = run_instance(inst, x)
        for bad in (0, 17):
            with pytest.raises(ie.IefwdError) as e:
                inst.set_stream_cache(bad)
            assert e.value.status == ie.EINVAL
        inst.set_stream_cache(4)
        places = [(32, 0), (64, 32), (96, 96)]
        for p in places:
            inst.prepare_quota(*p)
        for rep in range(2):
            for q, f in places:
                inst.set_quota(q, f)
                got = run_instance(inst, x)
                assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
                assert inst.get_cu_mask() == ie.build_cu_mask(256, 8, q, f)
        inst.set_stream_cache(1)
        got = run_instance(inst, x)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
        assert inst.get_cu_mask() == ie.build_cu_mask(256, 8, 96, 96)


@pytest.mark.parametrize("q", [40, 56, 64, 96])
def test_quota_spreads_over_shader_engines(q):
    # each XCD's share of a quota is spread over its shader engines as evenly as
    # it goes, and the workgroups of a launch are dealt to the engines in equal
    # numbers (whatever their CU counts): printed, the CU spread asserted
    shape = W.model_shape("encoder_l1_d128_s32_b2")
    with ie.Instance(**instance_config(shape, 1, 32)) as inst:
        inst.set_quota(q)
        run_instance(inst, W.make_input(1, 1, 32, 128))
        v = probe(inst.stream_handle(), 16384)
    xcc, se, cu = v[:, 0] & 0xF, (v[:, 1] >> 13) & 0x7, (v[:, 1] >> 8) & 0xF
    for x in range(8):
        sel = xcc == x
        cus = collections.defaultdict(set)
        wgs = collections.Counter()
        for s_, c_ in zip(se[sel].tolist(), cu[sel].tolist()):
            cus[s_].add(c_)
            wgs[s_] += 1
        n = [len(cus[k]) for k in sorted(cus)]
        if x == 0:
            print(f"quota {q}, XCD 0: CUs per engine {n}, workgroups per engine {[wgs[k] for k in sorted(wgs)]}",
                  flush=True)
        assert sum(n) == q // 8 and max(n) - min(n) <= 1
