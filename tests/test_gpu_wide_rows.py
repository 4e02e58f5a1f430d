"""Hidden sizes around the decode router's staging limit (d = 3584: seven
K steps per wavefront through its LDS regions; d = 4096 and 4352: rows read
in the fragment layout straight from memory) through the C ABI, at T = 1 and
16 (one-launch decode routing, stream path), and T = 600 (tile router and
tile path: 75 rows per expert); bf16 at all three, the 4-bit and the
quantized-expert mix at d = 4352.  Every token's output against the fp64
oracle (max-abs / max|ref| <= 1e-2) and the permutation against the
oracle's counting sort."""
import numpy as np
import pytest

import synth
from _gpu_helpers import device_layer, log, make_plan, oracle_compare, run_layer

pytestmark = pytest.mark.gpu

SHAPES = {f"d{d}_bf16": synth.Workload(f"wide_d{d}_bf16", 30 + i, synth.LayerShape(600, d, 32, 4, 128, "bf16"),
                                       prior="zipf", prior_param=1.1, tau=0.3)
          for i, d in enumerate((3584, 4096, 4352))}
# the quantized formats at d = 4352 (17 super-blocks, 34 blocks per quarter row: the narrowest chunking
# of their stream kernels)
SHAPES["d4352_q4"] = synth.Workload("wide_d4352_q4", 33, synth.LayerShape(600, 4352, 32, 4, 128, "q4b32"),
                                    prior="zipf", prior_param=1.1, tau=0.3)
SHAPES["d4352_kq"] = synth.Workload("wide_d4352_kq", 34, synth.LayerShape(600, 4352, 32, 4, 256, "kq"),
                                    prior="zipf", prior_param=1.1, tau=0.3)


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


@pytest.mark.parametrize("name", list(SHAPES))
def test_wide_rows(o, name):
    wl = SHAPES[name]
    li = synth.layer_inputs(wl)
    dl = device_layer(li)
    plan = make_plan(li, capacity=wl.shape.E)
    for T in (1, 16, 600):
        log(f"case {wl.name} T={T}")
        res = run_layer(plan, dl, T=T)
        assert res["status"] == 0
        err, near, _ = oracle_compare(o, li, res, list(range(T)), 1e-2)
        log(f"{wl.name} T={T} err={err:.3e} near_ties={len(near)}")
        counts, offsets, perm, inv = o.permute(np.sort(res["idx"], axis=1), wl.shape.E)
        assert np.array_equal(res["counts"], counts) and np.array_equal(res["offsets"], offsets)
        assert np.array_equal(res["perm"], perm) and np.array_equal(res["inv"], inv)
    # every expert is resident now: a forward that needs no fill, then one on the device work list
    for T in (1, 16):
        first = run_layer(plan, dl, T=T)
        direct = run_layer(plan, dl, T=T)
        assert direct["out"].cpu().numpy().tobytes() == first["out"].cpu().numpy().tobytes()
        err, near, _ = oracle_compare(o, li, direct, list(range(T)), 1e-2)
        log(f"{wl.name} T={T} device work list err={err:.3e} near_ties={len(near)}")
    plan.close()
