"""Lifecycle fault cells through the C ABI on the GPU, after the paper's fault
matrix (the table of prespecified fault modes in "Integrated Deterministic
Faults"): each cell names the invariant it exercises and checks the
required observation; every cell ends with a balanced terminal state (no fill
in flight, no busy window, no live consumer).

Faults are forced from the host (a bogus device generation word, a held
consumer, a fill of an object outside the manifest, a reset while a fill is
queued); no kernel is made to fault."""
import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, run_layer

pytestmark = pytest.mark.gpu

WL = synth.Workload("cells_bf16", 13, synth.LayerShape(40, 256, 12, 3, 128, "bf16"),
                    prior="dirichlet", prior_param=0.5, tau=0.4)


@pytest.fixture(scope="module")
def li():
    return synth.layer_inputs(WL)


@pytest.fixture(scope="module")
def control(li):
    """No-fault control: output of an all-resident plan."""
    dl = device_layer(li)
    plan = make_plan(li, capacity=12, per_window=4)
    out = run_layer(plan, dl)["out"].cpu().numpy()
    plan.close()
    return out


def balanced(plan):
    plan.poll()
    st = plan.stats()
    assert st["fills_in_flight"] == 0 and st["windows_busy"] == 0 and st["consumers_live"] == 0, st
    return st


def test_stale_generation_publishes_nothing(li, control):
    """Stale completion / wrong version: mismatch rejected before visibility,
    zero accepted outputs; the next forward refills and is exact."""
    import torch
    import paper_2608_23805_amd as msi
    log("cell stale_generation")
    dl = device_layer(li)
    plan = make_plan(li, capacity=12, per_window=4)
    res = run_layer(plan, dl)                                   # warm: every demanded expert resident
    demanded = np.nonzero(res["counts"])[0]
    slot = next(s for s in range(12) if plan.query(0, s).expert == int(demanded[0]))
    info = plan.query(0, slot)
    plan.debug_set_device_gen(0, slot, info.generation + 1000)
    canary = torch.full((WL.shape.T, WL.shape.d), 12345.0, device="cuda")
    res = run_layer(plan, dl, out=canary, check=False)
    assert res["status"] == msi.MSI_E_STALE
    assert torch.all(canary == 12345.0), "output written despite a stale slot"
    st = balanced(plan)
    assert st["stale_detected"] == 1
    res = run_layer(plan, dl)                                   # refilled, exact
    assert res["out"].cpu().numpy().tobytes() == control.tobytes()
    balanced(plan)
    plan.close()


def test_held_consumer_delays_reuse(li, control):
    """Held consumer: no reuse before consumers finish; full control-exact
    output and balanced release."""
    import paper_2608_23805_amd as msi
    log("cell held_consumer")
    dl = device_layer(li)
    plan = make_plan(li, capacity=3, per_window=4)             # 3 slots < demand: rounds, evictions
    t = plan.slot_fill(0, 5, slot=1)
    plan.poll()
    plan.hold(0, 1)
    with pytest.raises(msi.MsiError) as e:
        plan.slot_fill(0, 6, slot=1)
    assert e.value.status == msi.MSI_E_BUSY
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control.tobytes()
    info = plan.query(0, 1)
    assert info.expert == 5 and info.generation == t.generation and info.holds == 1   # never reused
    with pytest.raises(msi.MsiError) as e:
        plan.reset()                                            # reset with a live consumer
    assert e.value.status == msi.MSI_E_BUSY
    assert plan.destroy_status() == msi.MSI_E_BUSY              # shutdown with a live consumer
    plan.unhold(0, 1)
    balanced(plan)
    plan.close()


def test_wrong_object_rejected(li):
    """Wrong object: a request outside the manifest is rejected, and a forward
    demanding an object with no extent publishes nothing."""
    import torch
    import paper_2608_23805_amd as msi
    log("cell wrong_object")
    dl = device_layer(li)
    counts = run_layer(make_plan(li, capacity=12, per_window=4), dl)["counts"]
    missing = int(np.argmax(counts))                            # a demanded expert
    keep = [e for e in range(WL.shape.E) if e != missing]
    plan = make_plan(li, capacity=12, per_window=4, experts=keep)
    with pytest.raises(msi.MsiError) as e:
        plan.slot_fill(0, missing)
    assert e.value.status == msi.MSI_E_WRONG_OBJECT
    with pytest.raises(msi.MsiError) as e:
        plan.slot_fill(0, keep[0], slot=99)
    assert e.value.status == msi.MSI_E_WRONG_OBJECT
    canary = torch.full((WL.shape.T, WL.shape.d), -7.0, device="cuda")
    res = run_layer(plan, dl, out=canary, check=False)
    assert res["status"] == msi.MSI_E_WRONG_OBJECT
    assert torch.all(canary == -7.0)
    balanced(plan)
    plan.close()


def test_reset_with_inflight_fill(li, control):
    """Reset with outstanding work: the late completion does not publish; the
    next forward refills and is exact."""
    import torch
    log("cell reset_inflight")
    dl = device_layer(li)
    plan = make_plan(li, capacity=12, per_window=4)
    side = torch.cuda.Stream()
    t = plan.slot_fill(0, 2, side_stream=side)                  # queued, not yet observed
    plan.reset()
    torch.cuda.synchronize()
    plan.poll()
    info = plan.query(0, t.slot)
    assert info.state == 0 and info.expert == -1                # Vacant: never published
    st = plan.stats()
    assert st["fills_discarded"] == 1 and st["epoch"] == 1
    assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == control.tobytes()
    balanced(plan)
    plan.close()


def test_out_of_order_fills_exact(li, control):
    """Valid out-of-order completion: fills on two side streams in opposite
    orders complete in any order and the output stays control-exact."""
    import torch
    log("cell out_of_order")
    dl = device_layer(li)
    plan = make_plan(li, capacity=12, per_window=4)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for e in range(WL.shape.E):
        plan.slot_fill(0, e, side_stream=s1 if e % 2 else s2)
    torch.cuda.synchronize()
    plan.poll()
    st = plan.stats()
    assert st["fills_published"] == WL.shape.E
    out = run_layer(plan, dl)["out"].cpu().numpy()
    assert out.tobytes() == control.tobytes()
    assert plan.stats()["fills"] == WL.shape.E                  # everything was a hit
    balanced(plan)
    plan.close()


def test_stale_generation_on_device_work_list(li, control):
    """The same cell when the forward takes the device-built work list (all
    demanded experts published): nothing is published, then recovery."""
    import torch
    import paper_2608_23805_amd as msi
    log("cell stale_generation_direct")
    T = 12                                              # <= 16 tokens: stream path, device work list
    dl = device_layer(li)
    dl.x = dl.x[:T]
    plan = make_plan(li, capacity=12, per_window=4)
    ref = run_layer(plan, dl, T=T)                      # fills
    run_layer(plan, dl, T=T)                            # no fill: the next forward is eligible
    before = plan.stats()["hits"]
    res = run_layer(plan, dl, T=T)
    assert res["out"].cpu().numpy().tobytes() == ref["out"].cpu().numpy().tobytes()
    demanded = np.nonzero(res["counts"])[0]
    slot = next(s for s in range(12) if plan.query(0, s).expert == int(demanded[-1]))
    plan.debug_set_device_gen(0, slot, plan.query(0, slot).generation + 77)
    canary = torch.full((T, WL.shape.d), 3.5, device="cuda")
    bad = run_layer(plan, dl, T=T, out=canary, check=False)
    assert bad["status"] == msi.MSI_E_STALE and torch.all(canary == 3.5)
    again = run_layer(plan, dl, T=T)
    assert again["out"].cpu().numpy().tobytes() == ref["out"].cpu().numpy().tobytes()
    assert plan.stats()["hits"] > before
    balanced(plan)
    plan.close()


def test_explicit_fill_hit_keeps_generation(li):
    log("cell fill_hit")
    plan = make_plan(li, capacity=4, per_window=4)
    a = plan.slot_fill(0, 3)
    b = plan.slot_fill(0, 3)
    assert b.hit == 1 and b.slot == a.slot and b.generation == a.generation
    c = plan.slot_fill(0, 3, slot=(a.slot + 1) % 4)             # forced elsewhere: a new version
    assert c.hit == 0 and c.generation >= 1
    import torch
    torch.cuda.synchronize()
    balanced(plan)
    plan.close()


def _stale_tile_cell(li, capacity, persistent):
    """Stale generation on an expert of the tiled MFMA path: the forward
    returns MSI_E_STALE with the output untouched, and neither tile kernel
    wrote that expert's rows (its act and y rows keep a canary pattern while
    another tile-path expert's rows are overwritten), so both the gate/up
    tile check and the down tile check fired.  The next forward refills and
    is exact."""
    import torch
    import paper_2608_23805_amd as msi
    from _gpu_helpers import workspace_parts
    s = li.wl.shape
    dl = device_layer(li)
    plan = make_plan(li, capacity=capacity)
    ctrl = run_layer(plan, dl)
    counts, offsets = ctrl["counts"], ctrl["offsets"]
    tile = [e for e in range(s.E) if counts[e] > 16]
    row_tiles = sum((int(counts[e]) + 255) // 256 for e in tile) + (s.T + 255) // 256
    down_tiles, gu_tiles = row_tiles * (s.d // 256), row_tiles * (s.I // 128)
    log(f"stale tile cell: T={s.T} tile experts={len(tile)} gate/up tiles={gu_tiles} down tiles={down_tiles} "
        f"persistent={persistent}")
    assert (down_tiles > 256) == persistent and (gu_tiles > 256) == persistent, (gu_tiles, down_tiles)
    bad, other = tile[0], tile[-1]
    slot = next(q for q in range(capacity) if plan.query(0, q).expert == bad)
    plan.debug_set_device_gen(0, slot, plan.query(0, slot).generation + 1000)
    r = msi.Routing.alloc(s.T, s.K, s.E)
    ws = plan.workspace(s.T)
    cs = torch.cuda.current_stream()
    plan.route(dl.x, dl.wr, dl.bias, r, ws, cs)
    torch.cuda.synchronize()
    P = workspace_parts(s.T, s.E, s.K, s.d, s.I, s.wdtype)

    def rows(part, e, width):
        a = P[part] + int(offsets[e]) * width * 2
        return ws[a:a + int(counts[e]) * width * 2]
    for e in (bad, other):
        rows("act", e, s.I).fill_(0x5A)
        rows("y", e, s.d).fill_(0x5A)
    canary = torch.full((s.T, s.d), 6.25, device="cuda")
    st = plan.forward_status(0, dl.x, r, dl.shared, canary, ws, cs, torch.cuda.Stream())
    torch.cuda.synchronize()
    assert st == msi.MSI_E_STALE, st
    assert torch.all(canary == 6.25), "output written despite a stale slot"
    assert torch.all(rows("act", bad, s.I) == 0x5A), "gate/up tiles wrote rows of a stale slot"
    assert torch.all(rows("y", bad, s.d) == 0x5A), "down tiles wrote rows of a stale slot"
    assert not torch.all(rows("act", other, s.I) == 0x5A) and not torch.all(rows("y", other, s.d) == 0x5A)
    st = balanced(plan)
    assert st["stale_detected"] == 1
    again = run_layer(plan, dl)
    assert again["out"].cpu().numpy().tobytes() == ctrl["out"].cpu().numpy().tobytes()
    balanced(plan)
    plan.close()


def test_stale_generation_tile_path():
    """Tile path, down launch under one tile per CU (non-persistent kernel)."""
    log("cell stale_generation_tile")
    wl = synth.Workload("cells_tile_bf16", 19, synth.LayerShape(300, 512, 32, 4, 256, "bf16"),
                        prior="dirichlet", prior_param=0.5, tau=0.6)
    _stale_tile_cell(synth.layer_inputs(wl), capacity=32, persistent=False)


def test_stale_generation_persistent_tiles():
    """Prefill-shaped layer whose gate/up and down launches exceed one tile
    per CU, so both persistent tile kernels run (T = 4096, d = 2048, E = 16,
    K = 4)."""
    log("cell stale_generation_persistent")
    wl = synth.Workload("cells_persistent_bf16", 20, synth.LayerShape(4096, 2048, 16, 4, 512, "bf16"),
                        prior="dirichlet", prior_param=2.0, tau=0.2)
    _stale_tile_cell(synth.layer_inputs(wl), capacity=16, persistent=True)


QUANT_CELLS = {
    "q4_T1": ("q4b32", 1), "q4_T300": ("q4b32", 300), "kq_T12": ("kq", 12), "kq_T300": ("kq", 300),
}


@pytest.mark.parametrize("cell", sorted(QUANT_CELLS))
def test_stale_generation_quantized(cell):
    """Stale generation on the quantized kernels: the stream kernels of a
    device-built decode list (T = 1: the int4 kernels' token-0 path, whose
    generation compare comes after the work; T = 12 for the 4.5-bit mix) and
    the tile kernels of a device-built prefill list (T = 300).  The forward
    returns MSI_E_STALE with the output untouched and the stale expert's act
    and y rows unwritten while another expert's rows are overwritten; the
    next forward refills and is exact."""
    import torch
    import paper_2608_23805_amd as msi
    from _gpu_helpers import workspace_parts
    fmt, T = QUANT_CELLS[cell]
    wl = synth.Workload(f"cells_{cell}", 40 + sorted(QUANT_CELLS).index(cell),
                        synth.LayerShape(300, 512, 24, 4, 256, fmt), prior="dirichlet", prior_param=0.5, tau=0.4)
    li = synth.layer_inputs(wl)
    s = wl.shape
    log(f"cell stale_generation_quantized {cell}")
    dl = device_layer(li)
    plan = make_plan(li, capacity=s.E)
    run_layer(plan, dl, T=T)                                   # fills
    ref = run_layer(plan, dl, T=T)                             # no fill: the next forward takes a device-built list
    counts, offsets = ref["counts"], ref["offsets"]
    dem = [int(e) for e in np.nonzero(counts)[0]]
    bad = max(dem, key=lambda e: (int(counts[e]), -e))
    other = next(e for e in dem if e != bad)
    slot = next(q for q in range(s.E) if plan.query(0, q).expert == bad)
    plan.debug_set_device_gen(0, slot, plan.query(0, slot).generation + 1000)
    x = dl.x[:T]
    r = msi.Routing.alloc(T, s.K, s.E)
    ws = plan.workspace(T)
    cs = torch.cuda.current_stream()
    plan.route(x, dl.wr, dl.bias, r, ws, cs)
    torch.cuda.synchronize()
    P = workspace_parts(T, s.E, s.K, s.d, s.I, s.wdtype)

    def rows(part, e, width):
        a = P[part] + int(offsets[e]) * width * 2
        return ws[a:a + int(counts[e]) * width * 2]
    for e in (bad, other):
        rows("act", e, s.I).fill_(0x5A)
        rows("y", e, s.d).fill_(0x5A)
    canary = torch.full((T, s.d), 6.25, device="cuda")
    st = plan.forward_status(0, x, r, dl.shared, canary, ws, cs, torch.cuda.Stream())
    torch.cuda.synchronize()
    log(f"  T={T} bad expert {bad} ({int(counts[bad])} rows), other {other} ({int(counts[other])} rows): status {st}")
    assert st == msi.MSI_E_STALE, st
    assert torch.all(canary == 6.25), "output written despite a stale slot"
    assert torch.all(rows("act", bad, s.I) == 0x5A), "gate/up wrote rows of a stale slot"
    assert torch.all(rows("y", bad, s.d) == 0x5A), "down wrote rows of a stale slot"
    assert not torch.all(rows("act", other, s.I) == 0x5A) and not torch.all(rows("y", other, s.d) == 0x5A)
    assert balanced(plan)["stale_detected"] == 1
    again = run_layer(plan, dl, T=T)
    assert again["out"].cpu().numpy().tobytes() == ref["out"].cpu().numpy().tobytes()
    balanced(plan)
    plan.close()


def test_batch_limit_rejected():
    """A batch whose hidden states reach 2^31 bytes is rejected before any
    device work (the tile kernels address token rows with 32-bit offsets)."""
    import ctypes
    import torch
    import paper_2608_23805_amd as msi
    log("cell batch_limit")
    s = WL.shape
    li = synth.layer_inputs(WL)
    plan = make_plan(li, capacity=12, per_window=4)
    T = (1 << 31) // (s.d * 2)
    r = msi.Routing.alloc(1, s.K, s.E)
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    dummy = torch.empty(16, dtype=torch.int16, device="cuda")
    a = msi.msi_route_args(n_tokens=T, reserved=0, x=dummy.data_ptr(), w_router=dummy.data_ptr(), bias=None,
                           r=r.c(), workspace=ws.data_ptr(), workspace_bytes=ws.numel())
    assert msi.lib.msi_route(plan.h, ctypes.byref(a), None) == msi.MSI_E_INVALID_ARG
    assert "2^31" in msi.last_error()
    f = msi.msi_forward_args(layer=0, n_tokens=T, x=dummy.data_ptr(), r=r.c(), shared_object=None,
                             out=dummy.data_ptr(), workspace=ws.data_ptr(), workspace_bytes=ws.numel())
    assert msi.lib.msi_moe_forward(plan.h, ctypes.byref(f), None, None) == msi.MSI_E_INVALID_ARG
    balanced(plan)
    plan.close()
