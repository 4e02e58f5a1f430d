"""The decode fast path through the C ABI.

* One-launch routing (1 <= T <= 16 bf16 tokens) at an expert count that
  leaves the last router workgroup partly filled: selection against the fp64
  oracle, permutation and demanded-expert list bit-exact, and a second call
  on the same plan identical to the first (the launch's arrival counter is
  left at zero).
* A forward whose device-resolved work list meets a demanded expert without
  a published slot: the attempt publishes nothing, the forward is rescheduled
  on the host and still matches the oracle; the next two forwards of the
  same batch (all resident: host-built list, then the device path again) are
  byte-identical to it, so the status word was left clean.
* The same above the stream threshold (T > 16), where the four launch lists
  are built on the device.
"""
import dataclasses

import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, oracle_compare, run_layer

pytestmark = pytest.mark.gpu

TOL_BF16 = 1e-2

# E = 100: seven router workgroups, the last holding experts 96..99 only
ROUTE = synth.Workload("route_bf16", 15, synth.LayerShape(16, 256, 100, 8, 128, "bf16"),
                       prior="dirichlet", prior_param=0.5, tau=0.5)
# uniform routing over 64 experts: two 8-token batches demand different sets
MISS = synth.Workload("miss_bf16", 16, synth.LayerShape(16, 256, 64, 4, 128, "bf16"))


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


def _check_routing(o, res, E):
    idx = res["idx"]
    assert np.array_equal(idx, np.sort(idx, axis=1)), "idx not ascending"
    counts, offsets, perm, inv = o.permute(idx, E)
    assert np.array_equal(res["counts"], counts)
    assert np.array_equal(res["offsets"], offsets)
    assert np.array_equal(res["perm"], perm)
    assert np.array_equal(res["inv"], inv)
    demanded = np.nonzero(counts)[0]
    assert res["demand"][0] == len(demanded)
    assert np.array_equal(res["demand"][1:1 + len(demanded)], demanded)
    assert np.abs(res["w"].sum(axis=1) - 1.0).max() <= 1e-6


def test_decode_routing_partial_workgroup(o):
    li = synth.layer_inputs(ROUTE)
    for T in (1, 5, 16):
        log(f"case route_bf16 T={T}")
        lt = dataclasses.replace(li, x=li.x[:T])
        dl = device_layer(lt)
        plan = make_plan(li, capacity=ROUTE.shape.E)
        first = run_layer(plan, dl, T=T)
        oracle_compare(o, lt, first, list(range(T)), TOL_BF16)
        _check_routing(o, first, ROUTE.shape.E)
        again = run_layer(plan, dl, T=T)
        for k in ("idx", "w", "counts", "offsets", "perm", "inv", "logits"):
            assert again[k].tobytes() == first[k].tobytes(), k
        n = int(first["demand"][0])             # entries past the count are not written
        assert again["demand"][:1 + n].tobytes() == first["demand"][:1 + n].tobytes()
        assert again["out"].cpu().numpy().tobytes() == first["out"].cpu().numpy().tobytes()
        plan.close()


def test_device_work_list_miss_reschedules(o):
    li = synth.layer_inputs(MISS)
    la = dataclasses.replace(li, x=li.x[:8])
    lb = dataclasses.replace(li, x=li.x[8:16])
    da, db = device_layer(la), device_layer(lb)
    plan = make_plan(li, capacity=MISS.shape.E)
    log("case miss: batch a fills, then runs with no fill")
    ra = run_layer(plan, da, T=8)
    run_layer(plan, da, T=8)                       # no fill: the next forward tries the device path
    fills = plan.stats()["fills"]
    log("case miss: batch b on the device path meets unpublished experts")
    rb = run_layer(plan, db, T=8)
    new = set(np.nonzero(rb["counts"])[0]) - set(np.nonzero(ra["counts"])[0])
    assert new, "batch b demands no expert that batch a left unfilled"
    assert plan.stats()["fills"] == fills + len(new)
    oracle_compare(o, lb, rb, list(range(8)), TOL_BF16)
    _check_routing(o, rb, MISS.shape.E)
    log("case miss: batch b again, all resident (host list, then device list)")
    for _ in range(2):
        again = run_layer(plan, db, T=8)
        assert plan.stats()["fills"] == fills + len(new)
        assert again["out"].cpu().numpy().tobytes() == rb["out"].cpu().numpy().tobytes()
    plan.close()


# 96 tokens over 64 experts, skewed: popular experts take the tile path (more
# than 16 rows), rare ones the stream path
MISS_PRE = synth.Workload("miss_prefill_bf16", 24, synth.LayerShape(96, 256, 64, 4, 128, "bf16"),
                          prior="dirichlet", prior_param=0.3, tau=1.0)


def test_device_built_lists_above_stream_threshold(o):
    """T > 16: the work lists built on the device (after a forward that
    needed no fill) give byte-identical outputs to the host schedule, over
    both paths; a demanded expert without a published slot makes the
    attempt publish nothing and the forward is rescheduled on the host."""
    li = synth.layer_inputs(MISS_PRE)
    la = dataclasses.replace(li, x=li.x[:48])
    lb = dataclasses.replace(li, x=li.x[48:96])
    da, db = device_layer(la), device_layer(lb)
    plan = make_plan(li, capacity=MISS_PRE.shape.E)
    plan.set_timing(True, kinds=["permute"])       # the work-list kernel is the only launch of this kind
    log("case device lists: batch a fills, runs with no fill, then on the device lists")
    ra = run_layer(plan, da, T=48)
    c = ra["counts"]
    log(f"device lists: tile experts {(c > 16).sum()}, stream experts {((c > 0) & (c <= 16)).sum()}")
    assert (c > 16).any() and ((c > 0) & (c <= 16)).any()
    run_layer(plan, da, T=48)
    assert plan.timings()["permute"][0] == 0
    again = run_layer(plan, da, T=48)
    assert plan.timings()["permute"][0] == 1
    assert again["out"].cpu().numpy().tobytes() == ra["out"].cpu().numpy().tobytes()
    fills = plan.stats()["fills"]
    log("case device lists: batch b meets unpublished experts")
    rb = run_layer(plan, db, T=48)
    assert plan.timings()["permute"][0] == 2
    new = set(np.nonzero(rb["counts"])[0]) - set(np.nonzero(ra["counts"])[0])
    assert new and plan.stats()["fills"] == fills + len(new)
    oracle_compare(o, lb, rb, list(range(48)), TOL_BF16)
    _check_routing(o, rb, MISS_PRE.shape.E)
    for _ in range(2):
        again = run_layer(plan, db, T=48)
        assert again["out"].cpu().numpy().tobytes() == rb["out"].cpu().numpy().tobytes()
    assert plan.timings()["permute"][0] == 3
    plan.close()
