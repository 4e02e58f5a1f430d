"""Shared set-up of the GPU parity tests: inputs from ``synth`` copied into
pinned windows and device tensors, one route + forward through the C ABI, and
the comparison rules against the fp64 oracle."""
from __future__ import annotations

import dataclasses
import sys
from typing import Optional, Sequence

import numpy as np

import synth

NEAR_TIE = 1e-5          # oracle logit gap under which a different selection is accepted


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(a: np.ndarray, dtype: str):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


@dataclasses.dataclass
class DeviceLayer:
    li: synth.LayerInputs
    x: object
    wr: object
    bias: Optional[object]
    shared: Optional[object]


def device_layer(li: synth.LayerInputs) -> DeviceLayer:
    import torch
    s = li.wl.shape
    return DeviceLayer(
        li=li, x=to_device(li.x, s.xdtype), wr=to_device(li.wr, s.xdtype),
        bias=None if li.bias is None else torch.from_numpy(li.bias).cuda(),
        shared=None if li.shared is None else torch.from_numpy(li.shared).cuda())


def make_plan(li: synth.LayerInputs, capacity: int, transient: int = 8, per_window: int = 8,
              experts: Optional[Sequence[int]] = None):
    """Plan over one layer whose objects sit in pinned windows of
    ``per_window`` experts.  ``experts`` restricts the manifest."""
    import paper_2608_23805_amd as msi
    s = li.wl.shape
    ids = list(range(s.E)) if experts is None else list(experts)
    wins, entries = msi.pack_windows([li.expert(e) for e in ids], per_window, layer=0, expert_ids=ids)
    return msi.Plan(n_layers=1, n_experts=s.E, d_model=s.d, d_ff=s.I, top_k=s.K, wdtype=s.wdtype,
                    slots_per_layer=capacity, transient_slots=transient if capacity == 0 else 0,
                    windows=wins, objects=entries)


def run_layer(plan, dl: DeviceLayer, T: Optional[int] = None, compute=None, side=None, out=None,
              check=True):
    """route + forward; returns host copies of every output and the status."""
    import torch
    import paper_2608_23805_amd as msi
    s = dl.li.wl.shape
    T = s.T if T is None else T
    x = dl.x[:T]
    r = msi.Routing.alloc(T, s.K, s.E)
    ws = plan.workspace(T)
    if out is None:
        out = torch.empty((T, s.d), dtype=torch.float32, device="cuda")
    compute = compute or torch.cuda.current_stream()
    side = side or torch.cuda.Stream()
    plan.route(x, dl.wr, dl.bias, r, ws, compute)
    st = plan.forward_status(0, x, r, dl.shared, out, ws, compute, side)
    torch.cuda.synchronize()
    if check and st != 0:
        raise msi.MsiError(st, msi.last_error())
    L = ws[: T * s.E * 4].view(torch.float32).view(T, s.E)
    return {"status": st, "out": out, "idx": r.idx.cpu().numpy(), "w": r.weights.cpu().numpy(),
            "counts": r.counts.cpu().numpy(), "offsets": r.offsets.cpu().numpy(),
            "demand": r.demand.cpu().numpy(),
            "perm": r.perm.cpu().numpy(), "inv": r.inv.cpu().numpy(),
            "row_weight": r.row_weight.cpu().numpy(), "logits": L.cpu().numpy(), "routing": r}


def check_selection(gpu_idx: np.ndarray, ora: dict, tokens: Sequence[int]):
    """Selected sets must match exactly, except on tokens whose oracle top-K
    gap is below NEAR_TIE, where every differing expert must lie within
    NEAR_TIE of the K-th oracle logit.  Returns the list of accepted
    near-tie tokens."""
    near = []
    L = ora["logits"]
    for j, t in enumerate(tokens):
        g = np.sort(gpu_idx[t])
        o = ora["idx"][j]
        if np.array_equal(g, o):
            continue
        kth = np.sort(L[j])[::-1][len(o) - 1]
        diff = set(g.tolist()) ^ set(o.tolist())
        ok = ora["gap"][j] < NEAR_TIE and all(abs(L[j][e] - kth) < NEAR_TIE for e in diff)
        assert ok, f"token {t}: gpu {g} oracle {o} gap {ora['gap'][j]:.3e}"
        near.append(t)
    return near


def check_all_sets(o, li: synth.LayerInputs, gpu_idx: np.ndarray) -> dict:
    """Routed sets of every token against the oracle's fp64 logits and top-K
    (the near-tie rule of check_selection).  Returns the counts: tokens,
    exact matches, accepted near-tie differences, oracle near ties (top-K
    logit gap < NEAR_TIE), ties within 1e-4, and probability-gap near ties
    (restricted-softmax weight of the K-th expert within 1e-5 of the next
    expert's, both over the same normaliser)."""
    s = li.wl.shape
    L = o.router_logits(li.x, li.wr, li.bias, s.xdtype)
    idx, gap = o.select_topk(L, s.K)
    T = L.shape[0]
    g = np.sort(gpu_idx, axis=1)
    same = np.all(g == idx, axis=1)
    moved = []
    for t in np.nonzero(~same)[0]:
        kth = np.sort(L[t])[::-1][s.K - 1]
        diff = set(g[t].tolist()) ^ set(idx[t].tolist())
        ok = gap[t] < NEAR_TIE and all(abs(L[t][e] - kth) < NEAR_TIE for e in diff)
        assert ok, f"token {t}: gpu {g[t]} oracle {idx[t]} gap {gap[t]:.3e}"
        moved.append(int(t))
    srt = -np.sort(-L, axis=1)
    m = srt[:, :1]
    z = np.exp(srt[:, :s.K] - m).sum(axis=1)
    pgap = (np.exp(srt[:, s.K - 1] - m[:, 0]) - np.exp(srt[:, s.K] - m[:, 0])) / z
    return {"tokens": int(T), "exact": int(same.sum()), "near_tie_moved": len(moved), "moved_tokens": moved[:16],
            "oracle_near_ties_1e-5": int((gap < NEAR_TIE).sum()), "oracle_gaps_below_1e-4": int((gap < 1e-4).sum()),
            "prob_gap_below_1e-5": int((pgap < 1e-5).sum())}


def rel_err(a: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.abs(ref).max())
    return float(np.abs(np.asarray(a, np.float64) - ref).max() / (den if den > 0 else 1.0))


def oracle_compare(o, li: synth.LayerInputs, res: dict, tokens: Sequence[int], tol: float):
    """Oracle on ``tokens``; near-tie tokens are recomputed with the GPU's set.
    Returns (err, near_tie_tokens)."""
    s = li.wl.shape
    experts = [li.expert(e) for e in range(s.E)]
    ora = o.moe_layer(li.x, li.wr, li.bias, experts, li.shared, s.K, s.I, s.wdtype, s.xdtype,
                      tokens=tokens, want_logits=True)
    near = check_selection(res["idx"], ora, tokens)
    ref = ora["out"].copy()
    if near:
        pos = [list(tokens).index(t) for t in near]
        forced = np.sort(res["idx"][near], axis=1)
        r2 = o.moe_layer(li.x, li.wr, li.bias, experts, li.shared, s.K, s.I, s.wdtype, s.xdtype,
                         tokens=near, forced_idx=forced)
        ref[pos] = r2["out"]
    got = res["out"].cpu().numpy()[list(tokens)]
    err = rel_err(got, ref)
    assert err <= tol, f"max-abs/max|ref| {err:.3e} > {tol:.1e}"
    return err, near, ora


def workspace_parts(T: int, E: int, K: int, d: int, I: int, wdtype: str) -> dict:
    """Byte offsets of the workspace parts (the layout msi.h documents)."""
    a256 = lambda v: (v + 255) // 256 * 256  # noqa: E731
    ab = 4 if wdtype == "f32" else 2
    off, parts = 0, {}
    for name, n in (("logits", T * E * 4), ("blockhist", max((T + 255) // 256, 1) * E * 4),
                    ("act", T * K * I * ab), ("act_s", T * I * ab), ("y", T * K * d * ab), ("ys", T * d * ab)):
        parts[name] = off
        off += a256(n)
    parts["total"] = off
    return parts


def make_source_plan(li: synth.LayerInputs, capacity: int, path: str, n_windows: int = 8, inflight: int = 8,
                     transient: int = 8, seed: int = 0):
    """Plan over one layer whose expert objects are read from a canonical
    file (written here: gate, up and down of every expert as separate
    extents at shuffled, unaligned offsets) through ``n_windows`` staging
    windows with at most ``inflight`` reads in flight."""
    import paper_2608_23805_amd as msi
    s = li.wl.shape
    comps = synth.component_sizes(s)
    ext = synth.write_canonical_file(path, [li.expert(e) for e in range(s.E)], comps, seed=seed)
    extents = [(0, i, c, 0, off, n) for (i, c, off, n) in ext]
    wbytes = (s.object_bytes() + len(comps) * 8192 + 4095) // 4096 * 4096
    src = msi.Source([path], extents, n_windows=n_windows, window_bytes=wbytes, inflight=inflight)
    return msi.Plan(n_layers=1, n_experts=s.E, d_model=s.d, d_ff=s.I, top_k=s.K, wdtype=s.wdtype,
                    slots_per_layer=capacity, transient_slots=transient if capacity == 0 else 0,
                    windows=[], objects=[], source=src)
