"""msi_moe_forward_noalloc against msi_moe_forward through the C ABI.

Both entry points run the same forward on the same routing; the allocation-
free one keeps its act / y scratch in the library's static device array.
Outputs must be byte-identical (the entry points share every kernel), on
calls in a row with a smaller batch after a larger one, on the scheduled
path (T > 16, rounds and refills when the pool is smaller than the demand)
and on the device work list (T <= 16, every demanded expert resident).  A
batch needing more than the static scratch, or a passed workspace, is
rejected before any device work."""
import ctypes

import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan

pytestmark = pytest.mark.gpu

WL = synth.Workload("noalloc_bf16", 21, synth.LayerShape(300, 512, 32, 4, 256, "bf16"),
                    prior="dirichlet", prior_param=0.5, tau=0.6)


def _pair(plan, dl, T, label):
    import torch
    import paper_2608_23805_amd as msi
    s = dl.li.wl.shape
    x = dl.x[:T]
    cs = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    r = msi.Routing.alloc(T, s.K, s.E)
    ws = plan.workspace(T)
    plan.route(x, dl.wr, dl.bias, r, ws, cs)
    ref = torch.full((T, s.d), float("nan"), device="cuda")
    plan.forward(0, x, r, dl.shared, ref, ws, cs, side)
    got = torch.full((T, s.d), float("nan"), device="cuda")
    st = plan.forward_noalloc_status(0, x, r, dl.shared, got, cs, side)
    torch.cuda.synchronize()
    assert st == msi.MSI_OK, (label, msi.STATUS_NAMES.get(st), msi.last_error())
    a, b = ref.cpu().numpy(), got.cpu().numpy()
    assert np.isfinite(a).all()
    assert a.tobytes() == b.tobytes(), label
    log(f"noalloc {label} T={T}: byte-identical to msi_moe_forward")


def test_noalloc_matches_forward():
    li = synth.layer_inputs(WL)
    dl = device_layer(li)
    plan = make_plan(li, capacity=32)
    _pair(plan, dl, 300, "scheduled")
    _pair(plan, dl, 17, "scheduled, smaller")
    for T in (12, 12, 5):                        # all resident, no fill last time: device work list
        _pair(plan, dl, T, "device work list")
    plan.close()
    small = make_plan(li, capacity=5)            # rounds and refills
    _pair(small, dl, 300, "rounds")
    _pair(small, dl, 40, "rounds, smaller")
    small.close()


def test_noalloc_rejections():
    import torch
    import paper_2608_23805_amd as msi
    s = WL.shape
    li = synth.layer_inputs(WL)
    plan = make_plan(li, capacity=32)
    per_token = (s.K + 1) * (s.I + s.d) * 2
    T = msi.MSI_NOALLOC_SCRATCH_BYTES // per_token + 8
    r = msi.Routing.alloc(1, s.K, s.E)
    dummy = torch.empty(16, dtype=torch.float32, device="cuda")
    a = msi.msi_forward_args(layer=0, n_tokens=T, x=dummy.data_ptr(), r=r.c(), shared_object=None,
                             out=dummy.data_ptr(), workspace=None, workspace_bytes=0)
    assert msi.lib.msi_moe_forward_noalloc(plan.h, ctypes.byref(a), None, None) == msi.MSI_E_INVALID_ARG
    assert "scratch" in msi.last_error()
    ws = plan.workspace(1)
    a = msi.msi_forward_args(layer=0, n_tokens=1, x=dummy.data_ptr(), r=r.c(), shared_object=None,
                             out=dummy.data_ptr(), workspace=ws.data_ptr(), workspace_bytes=ws.numel())
    assert msi.lib.msi_moe_forward_noalloc(plan.h, ctypes.byref(a), None, None) == msi.MSI_E_INVALID_ARG
    assert "workspace" in msi.last_error()
    st = plan.stats()
    assert st["forwards"] == 0 and st["fills"] == 0
    plan.close()
