"""Exact ties in the router on the GPU, on each of the three selection paths
at E = 512, K = 10: T = 8 (one launch: logits, selection and permutation),
T = 100 (one-workgroup selection and permutation after the tile router) and
T = 512 (one wavefront per token, then the histogram / scan / scatter
permutation).

* A zero router (Wr = 0, b = 0, or b = +-0.0 alternating) makes every logit
  +0.0: the set must be experts {0..K-1} and every weight exactly
  float32(1/K).
* Router rows repeated across experts (expert e uses base row e mod 171, so
  each row appears three times, 171 ids apart: in different lanes and
  register slots of the selecting wavefront) make the logits of a group
  bitwise equal; the K-th place (10 = 3 + 3 + 3 + 1) falls inside a group on
  almost every token, and there the lower ids must win.  The oracle's
  sets are compared exactly; the only tolerated difference is a reported
  near tie between distinct groups (oracle logits that differ by less than
  1e-5 but are not equal).
* A full layer forward with a zero router routes every token to experts
  0..K-1 and matches the oracle.
"""
import numpy as np
import pytest

import synth
from _gpu_helpers import NEAR_TIE, device_layer, log, make_plan, oracle_compare, run_layer

pytestmark = pytest.mark.gpu

E, K, D = 512, 10, 512
PERIOD = 171


def _route_plan():
    import torch
    import paper_2608_23805_amd as msi
    win = torch.zeros(4096, dtype=torch.uint8, pin_memory=True)
    return msi.Plan(n_layers=1, n_experts=E, d_model=D, d_ff=128, top_k=K, wdtype="bf16", slots_per_layer=1,
                    windows=[win], objects=[])


def _route(plan, x_bits, wr_bits, bias):
    import torch
    import paper_2608_23805_amd as msi
    from _gpu_helpers import to_device
    T = x_bits.shape[0]
    r = msi.Routing.alloc(T, K, E)
    ws = plan.workspace(T)
    plan.route(to_device(x_bits, "bf16"), to_device(wr_bits, "bf16"),
               None if bias is None else torch.from_numpy(bias).cuda(), r, ws)
    torch.cuda.synchronize()
    return {k: getattr(r, k).cpu().numpy() for k in ("idx", "weights", "counts", "offsets", "demand", "perm",
                                                      "inv", "row_weight")}


def _check_perm(o, got):
    counts, offsets, perm, inv = o.permute(got["idx"], E)
    assert np.array_equal(got["counts"], counts) and np.array_equal(got["offsets"], offsets)
    assert np.array_equal(got["perm"], perm) and np.array_equal(got["inv"], inv)
    dem = np.nonzero(counts)[0]
    assert got["demand"][0] == len(dem) and np.array_equal(got["demand"][1:1 + len(dem)], dem)
    assert np.array_equal(got["row_weight"][inv.ravel()], got["weights"].ravel())


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


@pytest.fixture(scope="module")
def plan():
    p = _route_plan()
    yield p
    p.close()


@pytest.mark.parametrize("T", [8, 100, 512])
@pytest.mark.parametrize("bias_kind", ["none", "signed_zero"])
def test_zero_router_ties(o, plan, T, bias_kind):
    log(f"case ties zero_router T={T} bias={bias_kind}")
    x = synth.f32_to_bf16_bits(np.random.default_rng(T).standard_normal((T, D)).astype(np.float32))
    wr = np.zeros((E, D), dtype=np.uint16)
    bias = None
    if bias_kind == "signed_zero":
        bias = np.zeros(E, dtype=np.float32)
        bias[1::2] = -0.0
    got = _route(plan, x, wr, bias)
    assert np.all(got["idx"] == np.arange(K)[None, :])
    assert np.all(got["weights"] == np.float32(1.0 / K))
    L = o.router_logits(x, wr, bias, "bf16")
    idx, gap = o.select_topk(L, K)
    assert np.all(idx == np.arange(K)[None, :]) and np.all(gap == 0.0)
    _check_perm(o, got)


@pytest.mark.parametrize("T", [8, 100, 512])
def test_repeated_router_rows(o, plan, T):
    log(f"case ties repeated_rows T={T}")
    g = np.random.default_rng(1000 + T)
    base = (g.standard_normal((PERIOD, D)) * 0.02).astype(np.float32)
    wr = synth.f32_to_bf16_bits(base[np.arange(E) % PERIOD])
    x = synth.f32_to_bf16_bits(g.standard_normal((T, D)).astype(np.float32))
    # T = 100 adds a bias that is equal within each group
    bias = None if T != 100 else np.ascontiguousarray(
        (g.standard_normal(PERIOD).astype(np.float32) * 0.05)[np.arange(E) % PERIOD])
    got = _route(plan, x, wr, bias)
    L = o.router_logits(x, wr, bias, "bf16")
    idx, gap = o.select_topk(L, K)
    split, near = 0, []
    for t in range(T):
        srt = np.sort(L[t])[::-1]
        kth = srt[K - 1]
        if srt[K] == kth:
            split += 1                               # the K-th place falls inside a group of equal logits
        if np.array_equal(got["idx"][t], idx[t]):
            continue
        # the only accepted difference: a near tie between distinct logits
        assert 0.0 < gap[t] < NEAR_TIE, (t, got["idx"][t], idx[t], gap[t])
        diff = set(got["idx"][t].tolist()) ^ set(idx[t].tolist())
        assert all(abs(L[t][e] - kth) < NEAR_TIE for e in diff)
        near.append(t)
    log(f"ties repeated_rows T={T}: groups split at the K-th place on {split} tokens, near ties {len(near)}")
    assert split >= T // 2
    # equal logits get bitwise-equal weights; weights match the oracle's restricted softmax
    w_ref = o.gate_weights(L, got["idx"])
    assert np.abs(got["weights"] - w_ref).max() <= 2e-6
    for t in range(T):
        grp = got["idx"][t] % PERIOD
        for gv in np.unique(grp):
            ws = got["weights"][t][grp == gv]
            assert np.all(ws == ws[0]), (t, gv, ws)
    _check_perm(o, got)


def test_zero_router_forward(o):
    """Every token of a small layer routed to experts 0..K-1 by a zero router:
    four experts take all rows (tile path), the others none."""
    import dataclasses
    wl = synth.Workload("ties_small_bf16", 18, synth.LayerShape(300, 512, 32, 4, 256, "bf16"))
    li = synth.layer_inputs(wl)
    li = dataclasses.replace(li, wr=np.zeros_like(li.wr))
    log("case ties zero_router forward T=300 E=32")
    dl = device_layer(li)
    plan = make_plan(li, capacity=8)
    res = run_layer(plan, dl)
    assert np.all(res["idx"] == np.arange(4)[None, :])
    assert np.all(res["w"] == np.float32(0.25))
    assert np.array_equal(res["counts"][:4], [300] * 4) and not res["counts"][4:].any()
    err, near, _ = oracle_compare(o, li, res, list(range(0, 300, 7)) + [299], 1e-2)
    log(f"ties zero_router forward err={err:.3e}")
    plan.close()
