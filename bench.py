#!/usr/bin/env python3
"""Throughput of the slot-backed routed-expert MoE layer on one MI355X.

One step = one pass of the whole hot path over one batch: router logits,
top-K and restricted softmax, permutation, residency resolution (device-to-
host read of the per-expert counts, hits / misses / rounds), slot fills for
misses, the routed-expert gate/up and down projections, the shared expert,
and the fail-closed combine with its status read.

Headline (decode): T = 16 tokens, d = 2048, E = 512, top-10 + 1 shared
expert, intermediate 512, bf16 weights, fp32 router; all demanded experts
resident (512 slots), fresh hidden states each step (16 seeded batches in
rotation).  Secondary objects: the same decode with a 64-slot LRU pool
(fills over PCIe inside the step), and prefill T = 32768 with a
Dirichlet(0.3) router bias.  Every input is synthetic and seeded.

Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

METRIC = "routed tokens/sec per MoE layer (decode T=16, prefill T=32K); % HBM / MFMA peak"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
TIMING_PERIOD = 7               # decode: at most every 7th dominant-kernel launch carries events
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
# HBM traffic of the decode gate/up launch, from two hardware-counter runs
# (FETCH_SIZE, WRITE_SIZE) scaled by a plain copy kernel's counters; valid
# only while the kernel's sources hash to the recorded value
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "stream_gateup_decode_bf16_traffic.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_23805_amd", "csrc", f) for f in ("experts.hip", "common.h")]
# the same for the bf16 prefill gate/up launch (ring tile kernel)
PREFILL_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "ring_gemm_prefill_bf16_traffic.md")
PREFILL_KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_23805_amd", "csrc", f)
                          for f in ("gemm_ring.h", "tiles.hip", "common.h")]
# and for the quantized prefill gate/up tiles (int4; the k4 / k6 mix)
PREFILL_TRAFFIC_BY_FORMAT = {
    "bf16": (PREFILL_TRAFFIC_FILE, PREFILL_KERNEL_SOURCES),
    "q4b32": (os.path.join(ROOT, "profiles", "tile_q4_prefill_traffic.md"),
              [os.path.join(ROOT, "paper_2608_23805_amd", "csrc", f) for f in ("experts_q4.hip", "common.h")]),
    "kq": (os.path.join(ROOT, "profiles", "tile_kq_prefill_traffic.md"),
           [os.path.join(ROOT, "paper_2608_23805_amd", "csrc", f) for f in ("experts_kq.hip", "common.h")]),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _setup(wl, capacity, T=None, n_batches=1):
    import torch
    import synth
    import paper_2608_23805_amd as msi
    from _gpu_helpers import to_device
    s = wl.shape
    T = s.T if T is None else T
    t0 = time.time()
    li = synth.layer_inputs(wl)
    wins, entries = msi.pack_windows([li.expert(e) for e in range(s.E)], 8, layer=0)
    plan = msi.Plan(n_layers=1, n_experts=s.E, d_model=s.d, d_ff=s.I, top_k=s.K, wdtype=s.wdtype,
                    slots_per_layer=capacity, transient_slots=8 if capacity == 0 else 0,
                    windows=wins, objects=entries)
    xs = [to_device(synth.hidden_states(wl, 0, step, T), s.xdtype) for step in range(n_batches)]
    dev = dict(wr=to_device(li.wr, s.xdtype),
               bias=None if li.bias is None else torch.from_numpy(li.bias).cuda(),
               shared=torch.from_numpy(li.shared).cuda())
    r = msi.Routing.alloc(T, s.K, s.E)
    ws = plan.workspace(T)
    out = torch.empty((T, s.d), dtype=torch.float32, device="cuda")
    log(f"[bench] {wl.name}: set up in {time.time() - t0:.1f}s (capacity {capacity}, T {T})")
    return li, plan, xs, dev, r, ws, out


def _run(plan, xs, dev, r, ws, out, steps, warmup, cs, side, on_step=None):
    """warmup + timed steps; returns ms per step of the timed region.  Each
    step is msi_route then msi_moe_forward through argument structs built
    once per input buffer (the binding's prepare_step)."""
    import torch
    import paper_2608_23805_amd as msi
    calls = [plan.prepare_step(0, x, dev["wr"], dev["bias"], r, dev["shared"], out, ws, cs, side) for x in xs]

    def step(i):
        st = calls[i % len(calls)]()
        if st != 0:
            raise msi.MsiError(st, msi.last_error())
        if on_step is not None:
            on_step(i)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    plan.timings(reset=True)
    t0 = time.perf_counter()
    for i in range(steps):
        step(warmup + i)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / max(steps, 1)


def timing_period(steps):
    """Every how many steps the decode gate/up launch carries events: an odd
    period (coprime with the 16-batch rotation, so every batch is sampled),
    at most TIMING_PERIOD, and at least 6 timed launches when the run has
    that many steps (each timed launch adds host time to the step)."""
    p = max(1, min(TIMING_PERIOD, steps // 6))
    return p if p % 2 else p - 1


def bench_decode(args, cs, side):
    import synth
    wl = synth.WORKLOADS["decode_bf16"]
    s = wl.shape
    li, plan, xs, dev, r, ws, out = _setup(wl, capacity=512, n_batches=16)
    # warm-up fills every expert the rotation demands; the timed region then runs all-resident.
    # Telemetry: the dominant launch (gate/up) carries start / stop events that
    # the runtime records at the kernel's own start and end.  Each timed launch
    # costs host time on this latency-bound step, so only every
    # TIMING_PERIOD-th step of the timed region is timed (the period is
    # coprime with the 16 batches, so every batch is sampled).
    # (at least one pass over the whole rotation, whatever --warmup says, so the timed region needs no fill)
    _run(plan, xs, dev, r, ws, out, 0, max(args.warmup, len(xs)), cs, side)
    plan.set_timing(args.telemetry == "on", kinds=["gateup_stream"])
    period = timing_period(args.steps)
    plan.set_timing_period(period)
    before = plan.stats()
    ms = _run(plan, xs, dev, r, ws, out, args.steps, 0, cs, side)
    t = plan.timings()
    st = plan.stats()
    fills_timed = st["fills"] - before["fills"]
    if fills_timed:
        raise RuntimeError(f"decode: {fills_timed} fills inside the timed region of an all-resident run")
    # a further untimed pass with every launch carrying events: per-kernel durations
    plan.set_timing(args.telemetry == "on")
    plan.set_timing_period(1)
    _run(plan, xs, dev, r, ws, out, 32, 0, cs, side)      # _run clears the telemetry before its steps
    t_all = plan.timings()
    # algorithmic bytes of each step's gate/up launch (one round): the
    # demanded experts' Wg and Wu once, their tokens' x rows once, act written
    # once; the down launch reads Wd and act once and writes bf16 rows once
    bytes_b, down_b = [], []
    for b in range(len(xs)):
        plan.route(xs[b], dev["wr"], dev["bias"], r, ws, cs)
        c = r.counts.cpu().numpy()
        dem = c[c > 0]
        # the shared expert rides in the same launches: one more object, T more rows
        n_obj, n_rows = len(dem) + 1, int(dem.sum()) + s.T
        bytes_b.append(n_obj * 2 * s.I * s.d * 2 + n_rows * (s.d * 2 + s.I * 2))
        down_b.append(n_obj * s.d * s.I * 2 + n_rows * (s.I * 2 + s.d * 2))
    per_step_bytes = [bytes_b[i % len(xs)] for i in range(0, args.steps, period)]
    n_gu, ms_gu = t["gateup_stream"]
    n_dn, ms_dn = t_all["down_stream"]
    avg_gu = ms_gu / max(n_gu, 1)
    avg_dn = ms_dn / max(n_dn, 1)
    bytes_gu = sum(per_step_bytes) / max(len(per_step_bytes), 1)
    bytes_dn = sum(down_b[i % len(xs)] for i in range(32)) / 32
    achieved = bytes_gu / (avg_gu * 1e-3) / 1e9 if avg_gu > 0 else 0.0
    kernels = {k: {"launches": n, "avg_us": round(v * 1e3 / max(n, 1), 2)} for k, (n, v) in t_all.items() if n}
    plan.close()
    res = dict(ms=ms, T=s.T, tokens_per_s=s.T / (ms * 1e-3), kernels=kernels,
               roofline={"bound": "hbm", "kernel": "stream_gateup_kernel", "achieved": round(achieved, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": recorded_traffic(), "bytes_per_launch": int(bytes_gu),
                         "avg_launch_us": round(avg_gu * 1e3, 2), "launches_timed": n_gu,
                         "bytes_per_batch_mean": int(sum(bytes_b) / len(bytes_b))},
               down={"achieved_GBs": round(bytes_dn / (avg_dn * 1e-3) / 1e9, 1) if avg_dn > 0 else None,
                     "avg_launch_us": round(avg_dn * 1e3, 2), "bytes_per_launch": int(bytes_dn)},
               stats={k: st[k] for k in ("fills", "hits", "misses", "rounds")}, fills_in_timed_region=fills_timed)
    log(f"[bench] decode: {ms * 1e3:.1f} us/step, {res['tokens_per_s']:.0f} tok/s, gate/up {avg_gu * 1e3:.1f} us "
        f"= {achieved:.0f} GB/s, down {avg_dn * 1e3:.1f} us")
    return res, li


def bench_decode_lru(args, cs, side):
    import synth
    wl = synth.WORKLOADS["decode_bf16"]
    li, plan, xs, dev, r, ws, out = _setup(wl, capacity=64, n_batches=16)
    ms = _run(plan, xs, dev, r, ws, out, args.lru_steps, 4, cs, side)
    st = plan.stats()
    plan.close()
    res = dict(ms=round(ms, 3), tokens_per_s=round(wl.shape.T / (ms * 1e-3), 1), slots_per_layer=64,
               fills_per_step=round(st["fills"] / (args.lru_steps + 4), 1),
               h2d_GBs=round(st["h2d_bytes"] / (args.lru_steps + 4) / (ms * 1e-3) / 1e9, 1))
    log(f"[bench] decode LRU64: {ms:.2f} ms/step, {res['tokens_per_s']:.0f} tok/s")
    return res


def bench_prefill(args, cs, side, name="prefill_bf16"):
    import synth
    wl = synth.WORKLOADS[name]
    s = wl.shape
    li, plan, xs, dev, r, ws, out = _setup(wl, capacity=512, n_batches=1)
    # the timed steps carry no telemetry; a second pass with events around every launch gives the breakdown.
    # At least five untimed steps first: after the set-up's host work two were not enough for a steady state
    # (the timed bf16 steps then ran about 0.1 ms slower than the event pass that follows them)
    ms = _run(plan, xs, dev, r, ws, out, args.prefill_steps, max(args.warmup, 5), cs, side)
    plan.set_timing(True)
    ms_events = _run(plan, xs, dev, r, ws, out, args.prefill_steps, 0, cs, side)
    t = plan.timings()
    n_gu, ms_gu = t["gateup_tile"]
    avg_gu = ms_gu / max(n_gu, 1)
    c = r.counts.cpu().numpy()
    # rows taken by the tiled path (experts with more than 16 rows; the rest stream), plus the shared
    # expert's T rows, which ride in the same launch
    rows_tile = int(c[c > 16].sum()) + s.T
    flops_gu = 2.0 * rows_tile * s.d * 2 * s.I
    # algorithmic bytes of that launch: each tile expert's Wg and Wu (and the shared one's) once, every
    # token's x row once, act written once
    wbytes = gateup_weight_bytes(s)
    bytes_gu = (int((c > 16).sum()) + 1) * wbytes + s.T * s.d * 2 + rows_tile * s.I * 2
    layer_flops = 2.0 * s.T * (s.K * 3 * s.d * s.I + 3 * s.d * s.I + s.d * s.E)
    achieved = flops_gu / (avg_gu * 1e-3) / 1e12
    kernels = {k: {"launches": n, "avg_us": round(v * 1e3 / max(n, 1), 1)} for k, (n, v) in t.items() if n}
    routed_idx = r.idx.cpu().numpy()
    plan.close()
    res = dict(workload=name, value=round(s.T / (ms * 1e-3), 1), unit="routed tokens/s per layer",
               ms_per_step=round(ms, 3), ms_per_step_with_launch_events=round(ms_events, 3),
               kernel_sum_ms=round(sum(v for (n, v) in t.values()) / max(args.prefill_steps, 1), 3),
               T=s.T, layer_tflops=round(layer_flops / (ms * 1e-3) / 1e12, 1),
               layer_mfma_frac=round(layer_flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
               roofline={"bound": "mfma",
                         "kernel": {"q4b32": "tile_q4_kernel<GateUp>", "kq": "tile_kq_kernel<GateUp>"}.get(
                             s.wdtype, "ring_gemm_kernel<GateUp>"),
                         "achieved": round(achieved, 1),
                         "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
                         "traffic": recorded_traffic(*PREFILL_TRAFFIC_BY_FORMAT[s.wdtype]),
                         "flops_per_launch": flops_gu, "algorithmic_bytes_per_launch": bytes_gu,
                         "avg_launch_us": round(avg_gu * 1e3, 1),
                         "note": {"q4b32": "int4 weights unpacked to bf16 MFMA operands",
                                  "kq": "4.5-bit weights unpacked to exact bf16 MFMA operands, per-sub-block "
                                        "scale and min applied in fp32"}.get(s.wdtype, "")},
               kernels=kernels, _routed_idx=routed_idx)
    log(f"[bench] prefill: {ms:.3f} ms/step, {res['value']:.0f} tok/s, layer {res['layer_tflops']} TFLOP/s, "
        f"gate/up {avg_gu * 1e3:.0f} us = {achieved:.0f} TFLOP/s")
    return res


def gateup_weight_bytes(s):
    """Bytes of one expert's Wg and Wu in the layer's storage format."""
    if s.wdtype == "q4b32":
        return 2 * s.I * (s.d // 2 + s.d // 32 * 2)
    if s.wdtype == "kq":
        return 2 * s.I * (s.d // 2 + s.d // 256 * 16)
    return 2 * s.I * s.d * 2


def bench_decode_quant(args, cs, side, name):
    """Decode with quantized experts, all demanded experts resident:
    decode_q4 (T = 1, ~21 MB of weights per step, launch-bound) and
    decode_kq (T = 16).  A second, untimed pass with events on every launch
    gives the gate/up stream kernel's duration and its algorithmic bandwidth
    (the demanded experts' and the shared expert's Wg and Wu once, each routed
    row's x read and act written once)."""
    import synth
    wl = synth.WORKLOADS[name]
    s = wl.shape
    li, plan, xs, dev, r, ws, out = _setup(wl, capacity=512, n_batches=16)
    _run(plan, xs, dev, r, ws, out, 0, max(args.warmup, len(xs)), cs, side)
    before = plan.stats()
    ms = _run(plan, xs, dev, r, ws, out, args.steps, 0, cs, side)
    fills_timed = plan.stats()["fills"] - before["fills"]
    if fills_timed:
        plan.close()
        raise RuntimeError(f"{name}: {fills_timed} fills inside the timed region of an all-resident run")
    plan.set_timing(args.telemetry == "on")
    _run(plan, xs, dev, r, ws, out, 32, 0, cs, side)
    t = plan.timings()
    plan.set_timing(False)
    gu_bytes = []
    for b in range(len(xs)):
        plan.route(xs[b], dev["wr"], dev["bias"], r, ws, cs)
        c = r.counts.cpu().numpy()
        dem = c[c > 0]
        gu_bytes.append((len(dem) + 1) * gateup_weight_bytes(s) + (int(dem.sum()) + s.T) * (s.d * 2 + s.I * 2))
    plan.close()
    n_gu, ms_gu = t.get("gateup_stream", (0, 0.0))
    avg_gu = ms_gu / max(n_gu, 1)
    bytes_gu = sum(gu_bytes[i % len(xs)] for i in range(32)) / 32
    kernels = {k: {"launches": n, "avg_us": round(v * 1e3 / max(n, 1), 2)} for k, (n, v) in t.items() if n}
    res = dict(workload=name, T=s.T, ms=round(ms, 4), tokens_per_s=round(s.T / (ms * 1e-3), 1),
               fills_in_timed_region=fills_timed, kernels=kernels,
               gateup_stream={"avg_launch_us": round(avg_gu * 1e3, 2), "bytes_per_launch": int(bytes_gu),
                              "achieved_GBs": round(bytes_gu / (avg_gu * 1e-3) / 1e9, 1) if avg_gu > 0 else None,
                              "frac_of_hbm_peak": round(bytes_gu / (avg_gu * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
                              if avg_gu > 0 else None})
    log(f"[bench] {name}: {ms * 1e3:.1f} us/step, {res['tokens_per_s']:.0f} tok/s, gate/up {avg_gu * 1e3:.1f} us")
    return res


def h2d_peak_gbs(nbytes=1 << 30, reps=4):
    """Pinned host -> device copy bandwidth on this machine (one 1 GiB copy
    from page-locked memory per repetition, best of reps)."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    best = 0.0
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        best = max(best, nbytes / (time.perf_counter() - t0) / 1e9)
    del src, dst
    return best


def bench_stack(args, cs, side):
    """48-layer stack, T = 4096: one pass at capacities 0 and 64 (fills over
    PCIe every layer), a cold and a warm pass at 512 (all resident).  The
    overlap fraction of a pass with fills compares its wall W with copies
    alone, C = H2D bytes / measured pinned H2D peak, and compute alone, K =
    the warm all-resident pass: (C + K - W) / min(C, K), 1 when the smaller
    hides entirely under the larger, 0 when they run one after the other
    (or when W - C, the time beyond the copies, exceeds K: then the pass is
    bound by the copies and their overheads, and copy_efficiency = C / W says
    how close it comes to the copies alone)."""
    import time as _t
    import torch
    import synth
    from _stack import Stack
    wl = synth.WORKLOADS["stack_bf16"]
    pool = synth.layer_inputs(wl, layer=0)
    res = {"workload": "stack_bf16 (48 layers, T=4096, Zipf(1.1), windows of 8 experts)"}
    peak = h2d_peak_gbs()
    res["h2d_peak_GBs"] = round(peak, 1)
    for cap in (0, 64, 512):
        st = Stack(wl, capacity=cap, pool=pool)
        passes = 2 if cap == 512 else 1
        for p in range(passes):
            torch.cuda.synchronize()
            before = st.plan.stats()
            t0 = _t.perf_counter()
            st.run(compute=cs, side=side)
            dt = _t.perf_counter() - t0
            after = st.plan.stats()
            h2d = after["h2d_bytes"] - before["h2d_bytes"]
            key = f"capacity_{cap}" + ("_warm" if p == 1 else "")
            res[key] = {"ms": round(dt * 1e3, 1), "tokens_per_s_per_layer": round(wl.shape.T * st.L / dt, 1),
                        "fills": after["fills"] - before["fills"], "h2d_GB": round(h2d / 1e9, 2),
                        "h2d_GBs": round(h2d / dt / 1e9, 1)}
            log(f"[bench] stack {key}: {dt * 1e3:.0f} ms, H2D {h2d / dt / 1e9:.1f} GB/s")
        st.close()
        del st
        torch.cuda.empty_cache()
    K = res["capacity_512_warm"]["ms"] / 1e3
    for cap in (0, 64, 512):
        r = res[f"capacity_{cap}"]
        C = r["h2d_GB"] / peak
        W = r["ms"] / 1e3
        r["copy_alone_s"] = round(C, 3)
        r["overlap_fraction"] = round(max(0.0, (C + K - W) / min(C, K)), 3) if C > 0 else None
        r["h2d_frac_of_peak"] = round(r["h2d_GBs"] / peak, 3)
        # the pass beyond its copies at the measured peak: an upper bound on exposed compute
        # (K) plus per-copy and per-layer overheads; copy_efficiency = C / W
        r["beyond_copies_s"] = round(W - C, 3) if C > 0 else None
        r["copy_efficiency"] = round(C / W, 3) if C > 0 else None
    log(f"[bench] stack: pinned H2D peak {peak:.1f} GB/s, overlap "
        f"{[res[f'capacity_{c}']['overlap_fraction'] for c in (0, 64, 512)]}")
    return res


def bench_source_df(args, cs, side, pool=None):
    """The paper's matched source experiment on synthetic canonical files:
    a fixed decode workload (T = 16, fresh hidden states per step, E = 512,
    LRU64 per layer over several layers, each with its own router and bias)
    whose expert objects are read from one canonical file of 512
    Qwen3-Next-shaped objects (gate, up, down as three unaligned extents
    each), once with the blocking arm D (one staging window, one read in
    flight) and once with the asynchronous arm F (eight windows, eight reads
    in flight), in pairs of both orders.  Both arms must produce
    byte-identical outputs; reported: complete wall per arm, the F/D wall
    ratio, the time forwards waited on the source, reads and bytes."""
    import numpy as np
    import torch
    import synth
    import paper_2608_23805_amd as msi
    from _gpu_helpers import to_device
    wl = synth.WORKLOADS["stack_bf16"]
    s = wl.shape
    L, steps, T = args.df_layers, args.df_steps, 16
    t0 = time.time()
    if pool is None:
        pool = synth.layer_inputs(wl, layer=0)
    tmpdir = os.environ.get("TMPDIR", "/tmp")
    path = os.path.join(tmpdir, f"msi_canonical_{os.getpid()}.bin")
    comps = synth.component_sizes(s)
    objects = [pool.expert(e) for e in range(s.E)]
    # every arm reads a file written (and flushed) just for it, with the same bytes at the same offsets, so
    # no arm finds the extents in a read cache that an earlier arm filled
    ext = synth.write_canonical_file(path, objects, comps, seed=1, sync=True)
    loc = {}
    for (i, c, off, n) in ext:
        loc.setdefault(i, []).append((c, off, n))
    extents = []
    for l in range(L):
        m = synth.stack_expert_map(wl, l)
        for e in range(s.E):
            extents += [(l, e, c, 0, off, n) for (c, off, n) in loc[int(m[e])]]
    wbytes = (s.object_bytes() + 3 * 8192 + 4095) // 4096 * 4096
    wr = [to_device(synth.router_weight(wl, l), s.xdtype) for l in range(L)]
    bias = [torch.from_numpy(synth.router_bias(wl, l)).cuda() for l in range(L)]
    shared = [torch.from_numpy(synth.expert_object(wl, l, 0, shared=True)).cuda() for l in range(L)]
    xs = [to_device(synth.hidden_states(wl, 0, 100 + st, T), s.xdtype) for st in range(steps)]
    log(f"[bench] source D/F: canonical file {os.path.getsize(path) / 2**30:.2f} GiB, {L} layers x {steps} "
        f"decode steps, set up in {time.time() - t0:.1f}s")

    def arm(n_windows, inflight):
        src = msi.Source([path], extents, n_windows=n_windows, window_bytes=wbytes, inflight=inflight)
        plan = msi.Plan(n_layers=L, n_experts=s.E, d_model=s.d, d_ff=s.I, top_k=s.K, wdtype=s.wdtype,
                        slots_per_layer=64, windows=[], objects=[], source=src)
        r = msi.Routing.alloc(T, s.K, s.E)
        ws = plan.workspace(T)
        out = torch.empty((T, s.d), dtype=torch.float32, device="cuda")
        outs = []
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for st in range(steps):
            for l in range(L):
                plan.route(xs[st], wr[l], bias[l], r, ws, cs)
                plan.forward(l, xs[st], r, shared[l], out, ws, cs, side)
                outs.append(out.cpu().numpy().tobytes())
        torch.cuda.synchronize()
        wall = time.perf_counter() - t1
        stt, ss = plan.stats(), plan.source_stats()
        plan.close()
        return wall, outs, stt, ss

    pairs = []
    fresh = False                   # the file written above serves the first arm
    try:
        for order in ("DF", "FD")[:args.df_pairs]:
            res = {}
            for a in order:
                if fresh:
                    os.remove(path)
                    assert synth.write_canonical_file(path, objects, comps, seed=1, sync=True) == ext
                fresh = True
                res[a] = arm(1, 1) if a == "D" else arm(8, 8)
                log(f"[bench] source arm {a}: {res[a][0]:.2f} s, fills {res[a][2]['fills']}, "
                    f"waited {res[a][3]['wait_seconds']:.2f} s, peak depth {res[a][3]['peak_depth']}")
            assert res["D"][1] == res["F"][1], "D and F outputs differ"
            pairs.append((order, res["D"], res["F"]))
    finally:
        os.remove(path)
    d_w = [p[1][0] for p in pairs]
    f_w = [p[2][0] for p in pairs]
    ratio = float(np.exp(np.mean(np.log(np.array(f_w) / np.array(d_w)))))
    ss_f, ss_d, st_f = pairs[0][2][3], pairs[0][1][3], pairs[0][2][2]
    res = {"workload": f"decode T={T}, {L} layers x {steps} steps, LRU64 per layer, E=512, canonical file of "
                       f"512 objects x 3 extents", "pairs": [{"order": o, "D_s": round(d[0], 3), "F_s": round(f[0], 3),
                                                              "F_over_D": round(f[0] / d[0], 4)}
                                                             for o, d, f in pairs],
           "F_over_D_geomean": round(ratio, 4), "D_over_F": round(1 / ratio, 3),
           "outputs_identical": True, "fills_per_arm": st_f["fills"],
           "F_wait_s": round(ss_f["wait_seconds"], 3), "D_wait_s": round(ss_d["wait_seconds"], 3),
           "F_peak_depth": ss_f["peak_depth"], "D_peak_depth": ss_d["peak_depth"],
           "reads_per_arm": ss_f["reads_issued"], "logical_GB": round(ss_f["logical_bytes"] / 1e9, 2),
           "physical_GB": round(ss_f["physical_bytes"] / 1e9, 2),
           "F_read_GBs": round(ss_f["physical_bytes"] / min(f_w) / 1e9, 2),
           "direct_io": bool(ss_f["direct_files"]), "windows_free_at_end": True}
    log(f"[bench] source D/F: F/D wall {ratio:.3f} ({1 / ratio:.2f}x), D {d_w} s, F {f_w} s")
    return res


def kernel_sources_sha256(sources=None):
    import hashlib
    h = hashlib.sha256()
    for f in sources or KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(path=TRAFFIC_FILE, sources=None):
    """Measured HBM bytes per launch of the dominant kernel (decode gate/up by
    default), or None when no measurement exists or the kernel's sources
    changed since it was taken."""
    try:
        with open(path) as fh:
            kv = dict(re.findall(r"^([a-z0-9_]+): *(\S+)$", fh.read(), re.M))
    except OSError:
        return None
    if kv.get("kernel_sources_sha256") != kernel_sources_sha256(sources):
        return None
    try:
        return int(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration():
    """A plain copy of a known size (torch elementwise kernel: 1 GiB read,
    1 GiB written per launch), run under the same hardware counters as the
    decode kernel to scale FETCH_SIZE / WRITE_SIZE into bytes."""
    import torch
    n = 1 << 28
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(4):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read_per_launch": 4 * n, "bytes_written_per_launch": 4 * n,
                                           "launches": 4}}), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(li, budget_s, prefill_idx=None):
    """The fp64 oracle, as it stands, on the decode batch 0 (16 tokens), repeated
    until about budget_s seconds of wall time.  With ``prefill_idx`` (the
    GPU's routed sets of the 32K prefill batch) the oracle also routes that
    whole batch and the sets are compared, near ties counted."""
    import oracle
    s = li.wl.shape
    o = oracle.Oracle()
    experts = [li.expert(e) for e in range(s.E)]
    t0 = time.perf_counter()
    reps = 0
    while True:
        o.moe_layer(li.x, li.wr, li.bias, experts, li.shared, s.K, s.I, s.wdtype, s.xdtype)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    res = {"value": round(reps * s.T / el, 2), "unit": "routed tokens/s per layer", "cores": o.max_threads(),
           "cpu_model": cpu_model(), "kind": "oracle",
           "sample": f"decode layer T=16 (one seeded batch), {reps} repetitions, {el:.1f} s"}
    if prefill_idx is not None:
        import synth
        from _gpu_helpers import check_all_sets
        t1 = time.perf_counter()
        pli = synth.layer_inputs(synth.WORKLOADS["prefill_bf16"], lazy=True)
        res["prefill_routed_sets"] = check_all_sets(o, pli, prefill_idx)
        res["prefill_routed_sets"]["oracle_s"] = round(time.perf_counter() - t1, 1)
        log(f"[bench] prefill routed sets vs oracle: {res['prefill_routed_sets']}")
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--prefill-steps", type=int, default=10)
    ap.add_argument("--lru-steps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--telemetry", default="on", choices=["on", "off"],
                    help="HIP-event timing around each launch inside the decode timed region")
    ap.add_argument("--skip", default="", help="comma list of: prefill,lru,cpu,decode,q4,kq,stack,source")
    ap.add_argument("--df-layers", type=int, default=2, help="source D/F experiment: layers")
    ap.add_argument("--df-steps", type=int, default=6, help="source D/F experiment: decode steps")
    ap.add_argument("--df-pairs", type=int, default=2, help="source D/F experiment: pairs (1 or 2)")
    ap.add_argument("--only-source", action="store_true", help="run only the source D/F experiment")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB copy kernel (hardware-counter scale) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    skip = set(filter(None, args.skip.split(",")))
    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration()
        return
    cs = torch.cuda.current_stream()
    side = torch.cuda.Stream()

    if args.only_source:
        print(json.dumps({"source_df": bench_source_df(args, cs, side)}), flush=True)
        return
    if "decode" in skip:            # profiling aid: the prefill workloads only
        res = {}
        if "prefill" not in skip:
            res["prefill"] = bench_prefill(args, cs, side)
            res["prefill"].pop("_routed_idx")
        for fmt in ("q4", "kq"):
            if fmt not in skip:
                key = "prefill_q4" if fmt == "q4" else "prefill_kq"
                res[key] = bench_prefill(args, cs, side, key)
                res[key].pop("_routed_idx")
        print(json.dumps(res), flush=True)
        return
    dec, li = bench_decode(args, cs, side)
    extra = {}
    if "lru" not in skip:
        extra["decode_lru64"] = bench_decode_lru(args, cs, side)
    if "prefill" not in skip:
        extra["prefill"] = bench_prefill(args, cs, side)
    if "q4" not in skip:
        extra["prefill_q4"] = bench_prefill(args, cs, side, "prefill_q4")
        extra["decode_q4"] = bench_decode_quant(args, cs, side, "decode_q4")
    if "kq" not in skip:
        extra["prefill_kq"] = bench_prefill(args, cs, side, "prefill_kq")
        extra["decode_kq"] = bench_decode_quant(args, cs, side, "decode_kq")
    if "stack" not in skip:
        extra["stack"] = bench_stack(args, cs, side)
    if "source" not in skip:
        extra["source_df"] = bench_source_df(args, cs, side)
    pidx = extra["prefill"].pop("_routed_idx") if "prefill" in extra else None
    for key in ("prefill_q4", "prefill_kq"):
        if key in extra:
            extra[key].pop("_routed_idx")
    cpu = None if "cpu" in skip else cpu_baseline(li, args.cpu_seconds, pidx)

    s = li.wl.shape
    line = {
        "metric": METRIC, "value": round(dec["tokens_per_s"], 1), "unit": "routed tokens/s per layer",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(dec["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "decode_bf16 (Qwen3-Next-shaped MoE layer, all demanded experts resident)",
                   "T": s.T, "d": s.d, "E": s.E, "top_k": s.K, "d_ff": s.I, "shared_experts": 1,
                   "slots_per_layer": 512, "batches_in_rotation": 16},
        "roofline": dec["roofline"], "cpu_baseline": cpu,
        "fills_in_timed_region": dec["fills_in_timed_region"],
        "kernels_separate_pass": dec["kernels"], "down": dec["down"],
    }
    line.update(extra)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
