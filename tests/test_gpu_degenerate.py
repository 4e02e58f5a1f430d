"""The method's degenerate selections through the C ABI on every selection
path (T = 1 and 16: the one-launch decode router; T = 200: one-workgroup
selection; T = 600: one wavefront per token, then the histogram / scan /
scatter permutation):

* top-1 (K = 1, E = 64): every token's single expert carries weight exactly
  1 (the softmax over one selected logit);
* every expert selected (K = E = 16): each expert receives every token, the
  routing weights are the full softmax, and the layer is the dense mixture.

Every token's output against the fp64 oracle (max-abs / max|ref| <= 1e-2),
the permutation against the oracle's counting sort, and outputs
byte-identical between an all-resident plan and one with fewer slots than
experts (several rounds)."""
import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, oracle_compare, run_layer

pytestmark = pytest.mark.gpu

TOP1 = synth.Workload("top1_bf16", 28, synth.LayerShape(600, 256, 64, 1, 128, "bf16"),
                      prior="zipf", prior_param=1.1, tau=0.3)
DENSE = synth.Workload("dense_bf16", 29, synth.LayerShape(600, 256, 16, 16, 128, "bf16"))


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


@pytest.fixture(scope="module")
def layers():
    return {w.name: synth.layer_inputs(w) for w in (TOP1, DENSE)}


def _check(o, wl, li, T, caps):
    dl = device_layer(li)
    outs = []
    for cap in caps:
        log(f"case {wl.name} T={T} capacity={cap}")
        plan = make_plan(li, capacity=cap, per_window=16)
        res = run_layer(plan, dl, T=T)
        if cap == caps[0]:
            err, near, _ = oracle_compare(o, li, res, list(range(T)), 1e-2)
            log(f"{wl.name} T={T} err={err:.3e} near_ties={len(near)}")
            counts, offsets, perm, inv = o.permute(np.sort(res["idx"], axis=1), wl.shape.E)
            assert np.array_equal(res["counts"], counts) and np.array_equal(res["offsets"], offsets)
            assert np.array_equal(res["perm"], perm) and np.array_equal(res["inv"], inv)
            for _ in range(2):         # warm calls: the last one runs a device-built work list
                again = run_layer(plan, dl, T=T)
                assert again["out"].cpu().numpy().tobytes() == res["out"].cpu().numpy().tobytes()
        outs.append(res)
        plan.close()
    assert outs[0]["out"].cpu().numpy().tobytes() == outs[1]["out"].cpu().numpy().tobytes()
    return outs[0]


@pytest.mark.parametrize("T", [1, 16, 200, 600])
def test_top1(o, layers, T):
    res = _check(o, TOP1, layers[TOP1.name], T, (64, 12))
    assert np.all(res["w"] == 1.0), "a single selected expert carries weight exactly 1"


@pytest.mark.parametrize("T", [1, 16, 200, 600])
def test_every_expert_selected(o, layers, T):
    res = _check(o, DENSE, layers[DENSE.name], T, (16, 5))
    assert np.array_equal(res["idx"], np.tile(np.arange(16, dtype=res["idx"].dtype), (T, 1)))
    assert np.all(res["counts"] == T) and res["demand"][0] == 16
    assert np.all(np.abs(res["w"].sum(axis=1) - 1.0) <= 1e-6)
