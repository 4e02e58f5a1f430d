"""A stack of routed-expert layers with a residual stream (attention omitted),
driven through the C ABI: per layer route + forward, then h += out and
x = bf16(rmsnorm(h)) (all on the GPU).  Used by the stack test and the
benchmark.

Every layer has its own router weight, Zipf bias and shared expert; routed
expert objects come from one pool of E seeded objects through a seeded
per-layer permutation (``synth.stack_expert_map``), packed into pinned host
windows of 8 objects that all layers' manifest entries point into."""
from __future__ import annotations

import numpy as np

import synth
from _gpu_helpers import to_device


class Stack:
    def __init__(self, wl: synth.Workload, capacity: int, n_layers: int = None, per_window: int = 8,
                 pool: synth.LayerInputs = None, policy: str = "lru", prefetch_slots: int = 0):
        import torch
        import paper_2608_23805_amd as msi
        s = wl.shape
        self.wl, self.s = wl, s
        self.L = n_layers or wl.n_layers
        self.pool = pool or synth.layer_inputs(wl, layer=0)     # pool objects + layer 0's own tensors
        wins, entries0 = msi.pack_windows([self.pool.expert(e) for e in range(s.E)], per_window, layer=0)
        loc = {e: (w, o, n) for (_, e, w, o, n) in entries0}
        entries = []
        self.maps = []
        for l in range(self.L):
            m = synth.stack_expert_map(wl, l)
            self.maps.append(m)
            entries += [(l, e, *loc[int(m[e])]) for e in range(s.E)]
        self.plan = msi.Plan(n_layers=self.L, n_experts=s.E, d_model=s.d, d_ff=s.I, top_k=s.K,
                             wdtype=s.wdtype, slots_per_layer=capacity,
                             transient_slots=8 if capacity == 0 else 0, windows=wins, objects=entries,
                             policy=policy, prefetch_slots=prefetch_slots)
        self.prefetch_slots = prefetch_slots
        self.r_next = msi.Routing.alloc(s.T, s.K, s.E) if prefetch_slots else None
        self.wr, self.bias, self.shared = [], [], []
        for l in range(self.L):
            self.wr.append(to_device(synth.router_weight(wl, l), s.xdtype))
            self.bias.append(torch.from_numpy(synth.router_bias(wl, l)).cuda())
            self.shared.append(torch.from_numpy(synth.expert_object(wl, l, 0, shared=True)).cuda())
        self.x0 = to_device(self.pool.x, s.xdtype)
        self.r = msi.Routing.alloc(s.T, s.K, s.E)
        self.ws = self.plan.workspace(s.T)
        self.out = torch.empty((s.T, s.d), dtype=torch.float32, device="cuda")
        self.h = torch.empty((s.T, s.d), dtype=torch.float32, device="cuda")
        self.x = torch.empty_like(self.x0)

    def predict_next(self, l: int, compute):
        """Next-layer prediction for two-bank prefetch: layer l + 1's router on
        layer l's input; its demanded experts, most tokens first (ties by
        id), at most the prefetch bank's size, are prefetched into layer
        l + 1's bank while layer l runs."""
        import numpy as np
        self.plan.route(self.x, self.wr[l + 1], self.bias[l + 1], self.r_next, self.ws, compute)
        counts = self.r_next.counts.cpu().numpy()
        dem = np.nonzero(counts)[0]
        order = dem[np.lexsort((dem, -counts[dem]))]
        return [int(e) for e in order[:self.prefetch_slots]]

    def run(self, compute=None, side=None, capture=(), x0=None):
        """One pass over every layer; returns {layer: (x_l bf16, out_l, h_l,
        x_{l+1} bf16)} for the captured layers (host copies).  With a
        prefetch bank, each layer first prefetches the next layer's predicted
        experts.  x0: the stack's input (default: the workload's)."""
        import torch
        import paper_2608_23805_amd as msi
        compute = compute or torch.cuda.current_stream()
        side = side or torch.cuda.Stream()
        msi.residual_init(self.x0 if x0 is None else x0, self.h, self.x, compute)
        caps = {}
        for l in range(self.L):
            if self.prefetch_slots and l + 1 < self.L:
                self.plan.prefetch(l + 1, self.predict_next(l, compute), side)
            self.plan.route(self.x, self.wr[l], self.bias[l], self.r, self.ws, compute)
            self.plan.forward(l, self.x, self.r, self.shared[l], self.out, self.ws, compute, side)
            if l in capture:
                caps[l] = [self.x.cpu().numpy().view(np.uint16).copy(), self.out.cpu().numpy().copy(),
                           self.h.cpu().numpy().copy()]
            msi.residual_add(self.out, self.h, self.x, compute)
            if l in capture:
                caps[l].append(self.x.cpu().numpy().view(np.uint16).copy())
        torch.cuda.synchronize()
        return caps

    def layer_inputs(self, l: int, x_bf16: np.ndarray) -> synth.LayerInputs:
        """Oracle inputs of layer l on a given bf16 input (teacher forcing)."""
        wl, s = self.wl, self.s
        return synth.LayerInputs(
            wl=wl, layer=l, x=x_bf16, wr=synth.router_weight(wl, l), bias=synth.router_bias(wl, l),
            experts=[self.pool.expert(int(self.maps[l][e])) for e in range(s.E)],
            shared=synth.expert_object(wl, l, 0, shared=True))

    def close(self):
        self.plan.close()
