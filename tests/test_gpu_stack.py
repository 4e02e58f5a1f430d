"""Stacks of routed-expert MoE layers with a residual stream (attention
omitted), through the C ABI.

* The 48-layer stack (T = 4096, Zipf(1.1) popularity, windows of 8 experts,
  fills on a side stream): every captured layer output and the final
  residual stream are byte-identical at slot capacities 0 (zero-cache), 64
  and 512 per layer.  On every 8th layer (and the last), 16 sampled tokens
  match the fp64 oracle on that layer's own bf16 input (teacher forcing:
  routing amplifies rounding differences across layers), and the GPU's next
  layer input matches the oracle's residual step on the GPU's own stream.
* A reduced stack (6 layers, T = 64, d = 256, E = 16) is gated end to end:
  its final residual stream matches the oracle's stack within the bf16
  tolerance on every token whose routed sets agree with the oracle's at every
  layer; a token whose sets differ is accepted only when the oracle's top-K
  logit gap at the first differing layer is under 1e-3 (a near tie moved by
  the one-step bf16 rounding differences of that layer's input), and is
  counted and reported.
"""
import numpy as np
import pytest

import synth
from _gpu_helpers import log, oracle_compare

pytestmark = pytest.mark.gpu

CAPTURE = (0, 8, 16, 24, 32, 40, 47)
STACK_NEAR_TIE = 1e-3


def _check_residual(o, l, h_l, out_l, x_next):
    """The GPU's next-layer input against the oracle's residual step on the
    GPU's own h_l and out_l: within one half bf16 step of the fp64 value,
    except where the fp32 sum lands on the other side of a rounding point
    (then one full step)."""
    _, x_ref = o.residual_step(h_l.astype(np.float64), out_l.astype(np.float64))
    got = synth.bf16_bits_to_f32(x_next).astype(np.float64)
    ref = synth.bf16_bits_to_f32(x_ref).astype(np.float64)
    diff = np.abs(got - ref)
    assert np.all(diff <= np.abs(ref) * 2.0 ** -7 + 1e-30), f"residual stream at layer {l}"
    exact = float((x_next == x_ref).mean())
    log(f"stack layer {l}: next-layer input bit-equal to the oracle's on {exact:.6f} of elements")
    assert exact >= 0.999


def test_stack_capacities_and_teacher_forced_parity():
    import oracle
    import torch
    import paper_2608_23805_amd as msi
    from _gpu_helpers import to_device
    from _stack import Stack
    wl = synth.WORKLOADS["stack_bf16"]
    results = {}
    last = None
    for cap in (512, 64, 0):
        log(f"case stack_bf16 48 layers T=4096 capacity={cap}")
        st = Stack(wl, capacity=cap)
        caps = st.run(capture=CAPTURE)
        results[cap] = (st.h.cpu().numpy().tobytes(), {l: caps[l][1].tobytes() for l in CAPTURE})
        stats = st.plan.stats()
        log(f"stack capacity={cap}: fills={stats['fills']} hits={stats['hits']} rounds={stats['rounds']} "
            f"h2d_GB={stats['h2d_bytes'] / 1e9:.1f}")
        assert stats["fills_in_flight"] == 0 and stats["consumers_live"] == 0
        if last is None:
            last = (st, caps)
        else:
            st.close()
            del st
        torch.cuda.empty_cache()
    ref = results[512]
    for cap in (64, 0):
        assert results[cap][0] == ref[0], f"final residual differs at capacity {cap}"
        for l in CAPTURE:
            assert results[cap][1][l] == ref[1][l], f"layer {l} differs at capacity {cap}"
    st, caps = last
    o = oracle.Oracle()
    g = np.random.default_rng(9)
    for l in CAPTURE:
        x_l, out_l, h_l, x_next = caps[l]
        assert np.isfinite(h_l).all()
        _check_residual(o, l, h_l, out_l, x_next)
        li = st.layer_inputs(l, x_l)
        toks = sorted(g.choice(wl.shape.T, 16, replace=False).tolist())
        res = {"idx": None, "out": torch.from_numpy(out_l)}
        # the GPU selection for these tokens comes from re-routing layer l's input on the GPU
        r = msi.Routing.alloc(wl.shape.T, wl.shape.K, wl.shape.E)
        st.plan.route(to_device(x_l, "bf16"), st.wr[l], st.bias[l], r, st.ws)
        torch.cuda.synchronize()
        res["idx"] = r.idx.cpu().numpy()
        err, near, _ = oracle_compare(o, li, res, toks, 1e-2)
        log(f"stack layer {l}: teacher-forced err={err:.3e} over {len(toks)} tokens near_ties={len(near)}")
    st.close()


STACK_SMALL = synth.Workload("stack_small_bf16", 16, synth.LayerShape(64, 256, 16, 4, 128, "bf16"),
                             prior="zipf", prior_param=1.1, tau=0.3, n_layers=6)


def test_reduced_stack_end_to_end():
    import oracle
    import torch
    from _stack import Stack
    wl, s = STACK_SMALL, STACK_SMALL.shape
    log(f"case stack_small_bf16 {wl.n_layers} layers T={s.T} capacity=4 (rounds and refills every layer)")
    st = Stack(wl, capacity=4, per_window=4)
    caps = st.run(capture=tuple(range(wl.n_layers)))
    h_gpu = st.h.cpu().numpy().astype(np.float64)
    # the GPU's routed sets per layer (re-routing each captured input)
    import paper_2608_23805_amd as msi
    from _gpu_helpers import to_device
    gpu_idx = []
    for l in range(wl.n_layers):
        r = msi.Routing.alloc(s.T, s.K, s.E)
        st.plan.route(to_device(caps[l][0], "bf16"), st.wr[l], st.bias[l], r, st.ws)
        torch.cuda.synchronize()
        gpu_idx.append(np.sort(r.idx.cpu().numpy(), axis=1))
    o = oracle.Oracle()
    layers = []
    for l in range(wl.n_layers):
        li = st.layer_inputs(l, caps[l][0])
        layers.append(dict(wr=li.wr, bias=li.bias, experts=li.experts, shared=li.shared))
    h0 = synth.bf16_bits_to_f32(st.pool.x).astype(np.float64)
    ora = o.stack(h0, layers, s.K, s.I, s.wdtype)
    moved = []
    for t in range(s.T):
        for l in range(wl.n_layers):
            if not np.array_equal(gpu_idx[l][t], ora["idx"][l][t]):
                assert ora["gap"][l][t] < STACK_NEAR_TIE, (t, l, gpu_idx[l][t], ora["idx"][l][t], ora["gap"][l][t])
                moved.append((t, l))
                break
    keep = sorted(set(range(s.T)) - {t for t, _ in moved})
    den = np.abs(ora["h"]).max()
    err = float(np.abs(h_gpu[keep] - ora["h"][keep]).max() / den)
    min_gap = min(float(g.min()) for g in ora["gap"])
    log(f"stack_small end-to-end: max-abs/max|ref|={err:.3e} over {len(keep)} tokens; "
        f"tokens with a moved near tie: {len(moved)} {moved}; smallest oracle top-K gap {min_gap:.3e}")
    assert len(moved) <= s.T // 16
    assert err <= 1e-2
    st.close()
