"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bars: selected sets bit-exact except reported near-ties (oracle logit gap
< 1e-5), for every token also at T = 32768; max-abs / max|ref| <= 1e-5 for fp32 layers and <= 1e-2 for bf16
layers; permutation arrays bit-exact against the oracle's counting sort of
the GPU's own selection; outputs byte-identical across slot capacities.
"""
import dataclasses

import numpy as np
import pytest

import synth
from _gpu_helpers import (check_all_sets, device_layer, log, make_plan, oracle_compare, rel_err, run_layer)

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-5
TOL_BF16 = 1e-2


@pytest.fixture(scope="module")
def o():
    import oracle
    return oracle.Oracle()


def _check_permutation(o, res, E):
    counts, offsets, perm, inv = o.permute(np.sort(res["idx"], axis=1), E)
    assert np.array_equal(res["idx"], np.sort(res["idx"], axis=1)), "idx not ascending"
    assert np.array_equal(res["counts"], counts)
    assert np.array_equal(res["offsets"], offsets)
    demanded = np.nonzero(counts)[0]             # the demanded experts, ascending
    assert res["demand"][0] == len(demanded)
    assert np.array_equal(res["demand"][1:1 + len(demanded)], demanded)
    assert np.array_equal(res["perm"], perm)
    assert np.array_equal(res["inv"], inv)
    T, K = res["idx"].shape
    assert np.array_equal(res["row_weight"][inv.ravel()], res["w"].ravel())


def _check_weights(res, ora, tokens, tol=2e-6):
    assert np.all(np.abs(res["w"].sum(axis=1) - 1.0) <= 1e-6)
    for j, t in enumerate(tokens):
        if np.array_equal(np.sort(res["idx"][t]), ora["idx"][j]):
            assert np.abs(res["w"][t] - ora["w"][j]).max() <= tol, t


# ------------------------------------------------------------------ tiny fp32

TINY = synth.WORKLOADS["tiny_f32"]


@pytest.fixture(scope="module")
def tiny():
    return synth.layer_inputs(TINY)


def test_tiny_f32_layer(o, tiny):
    log("case tiny_f32 capacity=4")
    dl = device_layer(tiny)
    plan = make_plan(tiny, capacity=4, per_window=4)
    res = run_layer(plan, dl)
    toks = list(range(TINY.shape.T))
    err, near, ora = oracle_compare(o, tiny, res, toks, TOL_F32)
    log(f"tiny_f32 err={err:.3e} near_ties={len(near)}")
    _check_permutation(o, res, TINY.shape.E)
    _check_weights(res, ora, toks)
    # fp32 logits against the fp64 oracle
    assert np.abs(res["logits"] - ora["logits"]).max() <= 1e-5 * max(1.0, np.abs(ora["logits"]).max())
    st = plan.stats()
    assert st["rounds"] >= 4 and st["windows_busy"] == 0 and st["fills_in_flight"] == 0
    assert st["consumers_live"] == 0
    plan.close()


def test_tiny_capacity_bit_identity(tiny):
    dl = device_layer(tiny)
    outs = {}
    for cap in (0, 1, 4, 16):
        log(f"case tiny_f32 capacity={cap}")
        plan = make_plan(tiny, capacity=cap, transient=4, per_window=3)
        outs[cap] = run_layer(plan, dl)["out"].cpu()
        outs[(cap, 2)] = run_layer(plan, dl)["out"].cpu()      # second call: warm slots
        plan.close()
    ref = outs[16].numpy().tobytes()
    for k, v in outs.items():
        assert v.numpy().tobytes() == ref, k


# ------------------------------------------------------------------ small bf16 spanning tiles

SMALL = synth.Workload("small_bf16", 11, synth.LayerShape(300, 512, 32, 4, 256, "bf16"),
                       prior="dirichlet", prior_param=0.5, tau=0.6)


@pytest.fixture(scope="module")
def small():
    return synth.layer_inputs(SMALL)


def test_small_bf16_layer(o, small):
    log("case small_bf16 capacity=32")
    dl = device_layer(small)
    plan = make_plan(small, capacity=32)
    res = run_layer(plan, dl)
    counts = res["counts"]
    log(f"small_bf16 counts min={counts.min()} max={counts.max()} "
        f"stream={(counts[(counts > 0) & (counts <= 16)]).size} tile={(counts > 16).sum()}")
    assert (counts > 128).any() and ((counts > 0) & (counts <= 16)).any()   # both paths, several M tiles
    toks = list(range(SMALL.shape.T))
    err, near, ora = oracle_compare(o, small, res, toks, TOL_BF16)
    log(f"small_bf16 err={err:.3e} near_ties={len(near)}")
    _check_permutation(o, res, SMALL.shape.E)
    _check_weights(res, ora, toks)
    plan.close()


def test_small_bf16_capacity_bit_identity(small):
    dl = device_layer(small)
    ref = None
    for cap in (0, 5, 32):
        log(f"case small_bf16 capacity={cap}")
        plan = make_plan(small, capacity=cap, transient=6)
        for _ in range(3):               # at capacity 32 the third forward runs on device-built lists
            out = run_layer(plan, dl)["out"].cpu().numpy()
            if ref is None:
                ref = out
            assert out.tobytes() == ref.tobytes(), cap
        plan.close()


def test_small_bf16_ragged_T(o, small):
    """T = 1, 17, 129 (ragged tails of every tile shape) on the same layer."""
    for T in (1, 17, 129):
        log(f"case small_bf16 T={T}")
        li = dataclasses.replace(small, x=small.x[:T])
        dl = device_layer(li)
        plan = make_plan(small, capacity=32)
        res = run_layer(plan, dl, T=T)
        err, near, _ = oracle_compare(o, li, res, list(range(T)), TOL_BF16)
        _check_permutation(o, res, SMALL.shape.E)
        plan.close()


def test_empty_batch(small):
    """T = 0: routing writes zero counts, offsets and an empty demanded list
    (per-row arrays are empty, passed as null), the forward publishes nothing
    and returns MSI_OK, and the next full batch is unaffected."""
    import torch
    import paper_2608_23805_amd as msi
    log("case small_bf16 T=0")
    dl = device_layer(small)
    plan = make_plan(small, capacity=32)
    ref = run_layer(plan, dl)["out"].cpu().numpy()
    for _ in range(2):                            # after a full batch, and after an empty one
        res = run_layer(plan, dl, T=0)
        assert res["status"] == 0
        assert not res["counts"].any() and not res["offsets"].any() and res["demand"][0] == 0
        assert res["out"].shape == (0, SMALL.shape.d)
    st = plan.stats()
    assert st["fills_in_flight"] == 0 and st["consumers_live"] == 0
    assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == ref.tobytes()
    plan.close()


def test_stream_and_tile_paths_agree(small):
    """Forcing every expert through the tile path (threshold 1) changes only
    rounding, never more than the bf16 tolerance."""
    import paper_2608_23805_amd as msi
    dl = device_layer(small)
    plan = make_plan(small, capacity=32)
    a = run_layer(plan, dl)["out"].cpu().numpy()
    old = msi.stream_threshold()
    try:
        msi.stream_threshold(1)
        b = run_layer(plan, dl)["out"].cpu().numpy()
    finally:
        msi.stream_threshold(old)
    assert rel_err(b, a.astype(np.float64)) <= TOL_BF16
    plan.close()


# ------------------------------------------------------------------ full-size decode

DEC = synth.WORKLOADS["decode_bf16"]


@pytest.fixture(scope="module")
def dec():
    return synth.layer_inputs(DEC)


def test_decode_full_parity_and_capacities(o, dec):
    dl = device_layer(dec)
    outs = {}
    for cap in (512, 64, 0):
        log(f"case decode_bf16 capacity={cap}")
        plan = make_plan(dec, capacity=cap)
        res = run_layer(plan, dl)
        outs[cap] = res["out"].cpu().numpy()
        for _ in range(2):      # warm calls: at capacity 512 the last one runs the device work list
            again = run_layer(plan, dl)
            assert again["out"].cpu().numpy().tobytes() == outs[cap].tobytes()
        if cap == 512:
            toks = list(range(DEC.shape.T))
            err, near, ora = oracle_compare(o, dec, res, toks, TOL_BF16)
            log(f"decode err={err:.3e} near_ties={len(near)} demanded={(res['counts'] > 0).sum()}")
            _check_permutation(o, res, DEC.shape.E)
            _check_weights(res, ora, toks)
        st = plan.stats()
        log(f"decode capacity={cap} stats rounds={st['rounds']} fills={st['fills']} hits={st['hits']}")
        plan.close()
    assert outs[64].tobytes() == outs[512].tobytes()
    assert outs[0].tobytes() == outs[512].tobytes()


# ------------------------------------------------------------------ full-size prefill (all routed sets, sampled outputs)

PRE = synth.WORKLOADS["prefill_bf16"]


def test_prefill_full_sampled(o):
    li = synth.layer_inputs(PRE)
    dl = device_layer(li)
    log("case prefill_bf16 T=32768 capacity=512")
    plan = make_plan(li, capacity=512)
    res = run_layer(plan, dl)
    counts = res["counts"]
    log(f"prefill counts min={counts.min()} max={counts.max()} zero={(counts == 0).sum()}")
    _check_permutation(o, res, PRE.shape.E)
    assert np.all(np.abs(res["w"].sum(axis=1) - 1.0) <= 1e-6)
    # routed sets of all 32768 tokens against the oracle's selection
    sets = check_all_sets(o, li, res["idx"])
    log(f"prefill routed sets: {sets}")
    # outputs on a sample: first/last tokens, tokens of the rarest and busiest experts, every token whose
    # set moved on a near tie (the oracle recomputes those with the GPU's set)
    g = np.random.default_rng(7)
    rare = int(np.argmin(np.where(counts > 0, counts, 1 << 30)))
    busy = int(np.argmax(counts))
    toks = sorted(set([0, 1, PRE.shape.T - 1] + g.choice(PRE.shape.T, 96, replace=False).tolist()
                      + res["perm"][res["offsets"][rare]:res["offsets"][rare] + 8].tolist()
                      + res["perm"][res["offsets"][busy]:res["offsets"][busy] + 8].tolist()
                      + sets["moved_tokens"]))
    err, near, ora = oracle_compare(o, li, res, toks, TOL_BF16)
    log(f"prefill sampled {len(toks)} tokens err={err:.3e} near_ties={len(near)}")
    _check_weights(res, ora, toks)
    # all resident: the host schedule, then the device-built work lists, byte-identical
    for _ in range(2):
        assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == res["out"].cpu().numpy().tobytes()
    plan.close()


# ------------------------------------------------------------------ 4-bit block-quantized experts

SMALL_Q4 = synth.Workload("small_q4", 14, synth.LayerShape(260, 512, 24, 4, 256, "q4b32"),
                          prior="zipf", prior_param=1.5, tau=0.3)


@pytest.fixture(scope="module")
def small_q4():
    return synth.layer_inputs(SMALL_Q4)


def test_small_q4_layer_and_capacities(o, small_q4):
    dl = device_layer(small_q4)
    ref = None
    for cap in (24, 6, 0):
        log(f"case small_q4 capacity={cap}")
        plan = make_plan(small_q4, capacity=cap, transient=4)
        res = run_layer(plan, dl)
        for _ in range(2):               # at capacity 24 the last runs on device-built lists
            assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == res["out"].cpu().numpy().tobytes()
        if ref is None:
            counts = res["counts"]
            log(f"small_q4 counts min={counts.min()} max={counts.max()} "
                f"stream={((counts > 0) & (counts <= 16)).sum()} tile={(counts > 16).sum()}")
            assert (counts > 128).any() and ((counts > 0) & (counts <= 16)).any()
            toks = list(range(SMALL_Q4.shape.T))
            err, near, ora = oracle_compare(o, small_q4, res, toks, TOL_BF16)
            log(f"small_q4 err={err:.3e} near_ties={len(near)}")
            _check_permutation(o, res, SMALL_Q4.shape.E)
            ref = res["out"].cpu().numpy()
        else:
            assert res["out"].cpu().numpy().tobytes() == ref.tobytes(), cap
        plan.close()


def test_decode_q4_full(o):
    wl = synth.WORKLOADS["decode_q4"]
    li = synth.layer_inputs(wl)
    dl = device_layer(li)
    log("case decode_q4 T=1")
    outs = []
    for cap in (512, 0):
        plan = make_plan(li, capacity=cap)
        res = run_layer(plan, dl)
        if cap == 512:
            err, near, _ = oracle_compare(o, li, res, [0], TOL_BF16)
            log(f"decode_q4 err={err:.3e} near_ties={len(near)}")
            _check_permutation(o, res, wl.shape.E)
        for _ in range(2):      # warm calls: at capacity 512 the last one runs the device work list
            assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == res["out"].cpu().numpy().tobytes()
        outs.append(res["out"].cpu().numpy())
        plan.close()
    assert outs[0].tobytes() == outs[1].tobytes()


def test_prefill_q4_full_sampled(o):
    wl = synth.WORKLOADS["prefill_q4"]
    li = synth.layer_inputs(wl)
    dl = device_layer(li)
    log("case prefill_q4 T=32768 capacity=512")
    plan = make_plan(li, capacity=512)
    res = run_layer(plan, dl)
    counts = res["counts"]
    log(f"prefill_q4 counts min={counts.min()} max={counts.max()} zero={(counts == 0).sum()}")
    _check_permutation(o, res, wl.shape.E)
    sets = check_all_sets(o, li, res["idx"])
    log(f"prefill_q4 routed sets: {sets}")
    g = np.random.default_rng(8)
    busy = int(np.argmax(counts))
    toks = sorted(set([0, wl.shape.T - 1] + g.choice(wl.shape.T, 64, replace=False).tolist()
                      + res["perm"][res["offsets"][busy]:res["offsets"][busy] + 8].tolist()
                      + sets["moved_tokens"]))
    err, near, _ = oracle_compare(o, li, res, toks, TOL_BF16)
    log(f"prefill_q4 sampled {len(toks)} tokens err={err:.3e} near_ties={len(near)}")
    for _ in range(2):               # host schedule, then device-built work lists
        assert run_layer(plan, dl)["out"].cpu().numpy().tobytes() == res["out"].cpu().numpy().tobytes()
    plan.close()
