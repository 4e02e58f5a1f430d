"""A layer at the ABI's largest expert count and top-k (E = 1024, K = 16;
bf16, d = 256, I = 128) through the C ABI on every selection path: T = 1
(one launch, the one-token permutation) and T = 16 (one launch: logits,
selection and permutation; the device-built decode list on repeats), T = 200 (one-workgroup selection) and T = 600 (one
wavefront per token, then the histogram / scan / scatter permutation).  Every
token's output against the fp64 oracle (max-abs / max|ref| <= 1e-2), the
permutation against the oracle's counting sort, and outputs byte-identical at
capacity 1024 (one round) and 96 (several rounds)."""
import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, oracle_compare, run_layer

pytestmark = pytest.mark.gpu

WL = synth.Workload("limits_bf16", 27, synth.LayerShape(600, 256, 1024, 16, 128, "bf16"),
                    prior="zipf", prior_param=1.1, tau=0.3)


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


@pytest.fixture(scope="module")
def li():
    return synth.layer_inputs(WL)


@pytest.mark.parametrize("T", [1, 16, 200, 600])
def test_largest_expert_count_and_topk(o, li, T):
    dl = device_layer(li)
    outs = []
    for cap in (1024, 96):
        log(f"case limits E=1024 K=16 T={T} capacity={cap}")
        plan = make_plan(li, capacity=cap, per_window=64)
        res = run_layer(plan, dl, T=T)
        if cap == 1024:
            err, near, _ = oracle_compare(o, li, res, list(range(T)), 1e-2)
            log(f"limits T={T} err={err:.3e} near_ties={len(near)} demanded={int(res['demand'][0])}")
            counts, offsets, perm, inv = o.permute(np.sort(res["idx"], axis=1), WL.shape.E)
            assert np.array_equal(res["counts"], counts) and np.array_equal(res["offsets"], offsets)
            assert np.array_equal(res["perm"], perm) and np.array_equal(res["inv"], inv)
            for _ in range(2):                      # all resident: the device-built lists
                assert run_layer(plan, dl, T=T)["out"].cpu().numpy().tobytes() == \
                    res["out"].cpu().numpy().tobytes()
        outs.append(res["out"].cpu().numpy())
        plan.close()
    assert outs[0].tobytes() == outs[1].tobytes()
