"""Plans whose expert objects are read from canonical files by the bounded
source service (the Design section's "Bounded Source Service", "Stable Slots
and Bundle Publication" and "Separate Window and GPU-Slot Lifecycles"),
through the C ABI on the GPU.

* Outputs are byte-identical to those of a plan over always-resident host
  windows, at every capacity (all resident, rounds with refills, zero-cache)
  and for both source arms: one window with one read in flight (blocking)
  and eight windows with eight reads in flight (asynchronous).  Every object
  is a bundle of three extents (gate, up, down) at shuffled, unaligned file
  offsets, read with block-aligned covering reads.
* The remaining cells of the paper's fault-mode table ("Integrated
  Deterministic Faults"), forced from the host: a short read, EIO, a failed
  extent inside a bundle, a late stale completion after a newer fill of the
  same slot, reset with outstanding source work, shutdown with a read in
  flight, and valid out-of-order completions.  Fatal cells publish nothing
  (the output keeps its canary, the slot never becomes ready, no copy is
  made from the failed window); recoverable cells stay control-exact; every
  cell ends balanced (no fill or read in flight, every window Free, no live
  consumer).
"""
import os

import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, make_source_plan, run_layer

pytestmark = pytest.mark.gpu

WL = synth.Workload("source_bf16", 22, synth.LayerShape(300, 512, 32, 4, 256, "bf16"),
                    prior="dirichlet", prior_param=0.5, tau=0.6)


@pytest.fixture(scope="module")
def li():
    return synth.layer_inputs(WL)


@pytest.fixture(scope="module")
def control(li):
    dl = device_layer(li)
    plan = make_plan(li, capacity=32)
    out = {T: run_layer(plan, dl, T=T)["out"].cpu().numpy() for T in (300, 12)}
    plan.close()
    return out


def poll_until(plan, cond, seconds=20.0):
    """Poll the plan until cond() holds (the source's reads run on its own
    worker threads); False if it never does within the time limit."""
    import time
    t0 = time.time()
    while time.time() - t0 < seconds:
        plan.poll()
        if cond():
            return True
        time.sleep(0.005)
    return False


def balanced(plan):
    plan.poll()
    st, ss = plan.stats(), plan.source_stats()
    assert st["fills_in_flight"] == 0 and st["windows_busy"] == 0 and st["consumers_live"] == 0, st
    assert ss["windows_busy"] == 0 and ss["reads_completed"] == ss["reads_issued"], ss
    return st, ss


@pytest.mark.parametrize("arm", ["blocking_1x1", "async_8x8"])
def test_source_plan_matches_window_plan(li, control, tmp_path, arm):
    n_windows, inflight = (1, 1) if arm == "blocking_1x1" else (8, 8)
    dl = device_layer(li)
    for cap in (32, 5, 0):
        log(f"case source {arm} capacity={cap}")
        plan = make_source_plan(li, cap, str(tmp_path / f"canon_{cap}.bin"), n_windows=n_windows,
                                inflight=inflight, transient=6)
        for _ in range(2):
            out = run_layer(plan, dl)["out"].cpu().numpy()
            assert out.tobytes() == control[300].tobytes(), (arm, cap)
        for _ in range(3):                           # T <= 16: the device work list once nothing is filled
            out = run_layer(plan, dl, T=12)["out"].cpu().numpy()
            assert out.tobytes() == control[12].tobytes(), (arm, cap)
        st, ss = balanced(plan)
        log(f"source {arm} capacity={cap}: fills={st['fills']} reads={ss['reads_issued']} "
            f"peak_depth={ss['peak_depth']} logical={ss['logical_bytes']} physical={ss['physical_bytes']} "
            f"direct={ss['direct_files']} buffered={ss['buffered_files']} wait={ss['wait_seconds']:.3f}s")
        assert 1 <= ss["peak_depth"] <= inflight
        assert ss["reads_issued"] == 3 * st["fills"] and ss["requests_ready"] == st["fills"]
        assert ss["physical_bytes"] >= ss["logical_bytes"] == st["fills"] * WL.shape.object_bytes()
        assert ss["requests_failed"] == 0
        plan.close()


def _fatal_forward(plan, dl, expect):
    """A forward whose fill fails: the given status, out untouched."""
    import torch
    import paper_2608_23805_amd as msi
    canary = torch.full((WL.shape.T, WL.shape.d), 42.0, device="cuda")
    res = run_layer(plan, dl, out=canary, check=False)
    assert res["status"] == expect, (msi.STATUS_NAMES.get(res["status"]), msi.last_error())
    assert torch.all(canary == 42.0), "output written although a fill failed"
    return res


def _demanded(res):
    return [int(e) for e in np.nonzero(res["counts"])[0]]


@pytest.mark.parametrize("mode,component,expect", [("short", 0, -2), ("eio", 2, -9), ("short", 1, -2)],
                         ids=["short_read", "eio", "failed_extent_in_bundle"])
def test_source_fatal_cells(li, control, tmp_path, mode, component, expect):
    """Short read; EIO; failed bundle extent: publish only after complete
    valid movement -- zero accepted outputs, no readiness, no copy from the
    failed window; the executor drains; the next forward is exact."""
    log(f"cell source {mode} component={component}")
    dl = device_layer(li)
    plan = make_source_plan(li, 32, str(tmp_path / "canon.bin"))
    probe = run_layer(make_plan(li, capacity=32), dl)
    victim = _demanded(probe)[3]
    plan.source_fault(0, victim, component, mode)
    _fatal_forward(plan, dl, expect)
    st, ss = balanced(plan)
    assert ss["requests_failed"] == 1 and ss["reads_failed"] == 1
    for q in range(32):                              # the failed object never became ready anywhere
        info = plan.query(0, q)
        assert not (info.expert == victim and info.state in (2, 3, 4)), info
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control[300].tobytes()
    balanced(plan)
    plan.close()


def test_source_short_file(li, tmp_path):
    """A real short read: the canonical file loses its tail after the plan
    was created, so the extents there read short."""
    log("cell source truncated_file")
    dl = device_layer(li)
    path = str(tmp_path / "canon.bin")
    plan = make_source_plan(li, 32, path)
    os.truncate(path, os.path.getsize(path) // 3)
    _fatal_forward(plan, dl, -2)
    st, ss = balanced(plan)
    assert ss["requests_failed"] >= 1
    plan.close()


def test_source_late_stale_completion(li, control, tmp_path):
    """Late stale completion: the read of a fill still in flight when a newer
    fill of the same slot is requested completes late and is rejected; the
    slot keeps the newer version; the next forward is exact."""
    import torch
    log("cell source late_stale")
    dl = device_layer(li)
    plan = make_source_plan(li, 32, str(tmp_path / "canon.bin"))
    side = torch.cuda.Stream()
    plan.source_fault(0, 5, 0, "hold")
    old = plan.slot_fill(0, 5, slot=2, side_stream=side)      # held in the source
    new = plan.slot_fill(0, 6, slot=2, side_stream=side)      # newer fill of the same slot
    assert new.generation == old.generation + 1
    assert poll_until(plan, lambda: plan.query(0, 2).state == 2)
    info = plan.query(0, 2)
    assert info.expert == 6 and info.generation == new.generation and info.state == 2, info
    plan.source_release()                                      # the old read completes now, late
    assert poll_until(plan, lambda: plan.source_stats()["requests_stale"] >= 1)
    ss = plan.source_stats()
    assert ss["requests_stale"] == 1, ss
    info = plan.query(0, 2)
    assert info.expert == 6 and info.generation == new.generation, info
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control[300].tobytes()
    st, _ = balanced(plan)
    assert st["fills_discarded"] >= 1
    plan.close()


def test_source_reset_with_outstanding_read(li, control, tmp_path):
    """Reset with outstanding source work: the held read completes after the
    epoch advanced and publishes nothing; the slot is Vacant; exact after."""
    import torch
    log("cell source reset_outstanding")
    dl = device_layer(li)
    plan = make_source_plan(li, 32, str(tmp_path / "canon.bin"))
    plan.source_fault(0, 9, 1, "hold")
    t = plan.slot_fill(0, 9, side_stream=torch.cuda.Stream())
    plan.reset()
    plan.source_release()
    assert poll_until(plan, lambda: plan.source_stats()["requests_stale"] >= 1)
    info = plan.query(0, t.slot)
    assert info.state == 0 and info.expert == -1, info
    st, ss = balanced(plan)
    assert ss["requests_stale"] == 1 and st["fills_discarded"] == 1 and st["epoch"] == 1
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control[300].tobytes()
    balanced(plan)
    plan.close()


def test_source_shutdown_with_read_in_flight(li, tmp_path):
    """Shutdown with outstanding source work: destroy lets the held read go,
    drains the executor and returns (no wait for the hold's time limit)."""
    import time
    import torch
    log("cell source shutdown_outstanding")
    plan = make_source_plan(li, 32, str(tmp_path / "canon.bin"))
    plan.source_fault(0, 3, 2, "hold")
    plan.slot_fill(0, 3, side_stream=torch.cuda.Stream())
    assert plan.source_stats()["windows_busy"] == 1
    t0 = time.time()
    plan.close()
    assert time.time() - t0 < 10.0


def test_source_out_of_order_completion(li, control, tmp_path):
    """Valid out-of-order completion: the first of several explicit fills is
    held while the later ones complete; all publish, the output is exact."""
    import torch
    log("cell source out_of_order")
    dl = device_layer(li)
    plan = make_source_plan(li, 32, str(tmp_path / "canon.bin"))
    side = torch.cuda.Stream()
    plan.source_fault(0, 0, 0, "hold")
    for e in range(6):
        plan.slot_fill(0, e, side_stream=side)
    assert poll_until(plan, lambda: sum(plan.query(0, q).state == 2 for q in range(32)) >= 5)
    assert sum(plan.query(0, q).state == 2 for q in range(32)) == 5
    plan.source_release()
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control[300].tobytes()
    st, ss = balanced(plan)
    assert st["fills_published"] >= 6 and ss["requests_failed"] == 0
    plan.close()
