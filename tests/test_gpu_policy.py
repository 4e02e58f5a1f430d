"""Replacement policies and two-bank next-layer prefetch on a decode-shaped
stack (8 layers, T = 8 tokens per step, E = 64, K = 6, 16 slots per layer,
Zipf(1.1) popularity, 6 decode steps with fresh inputs), through the C ABI:
the output of every step is byte-identical under LRU, protected LRU and
either with a 6-slot prefetch bank (the policy moves bytes, never the
result); prefetched objects are used by the forwards; the protected policy
keeps more hits than plain LRU would lose to single-use objects."""
import numpy as np
import pytest

import synth
from _gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu

WL = synth.Workload("policy_bf16", 23, synth.LayerShape(8, 512, 64, 6, 256, "bf16"),
                    prior="zipf", prior_param=1.1, tau=0.3, n_layers=8)
STEPS = 6


def _run(policy, prefetch_slots, pool):
    import torch
    from _stack import Stack
    st = Stack(WL, capacity=16, per_window=8, pool=pool, policy=policy, prefetch_slots=prefetch_slots)
    outs = []
    for step in range(STEPS):
        x0 = to_device(synth.hidden_states(WL, 0, 50 + step), "bf16")
        st.run(x0=x0)
        outs.append(st.h.cpu().numpy().tobytes())
    torch.cuda.synchronize()
    stats = st.plan.stats()
    st.close()
    return outs, stats


def test_policies_and_prefetch_are_output_exact():
    pool = synth.layer_inputs(WL, layer=0)
    runs = {}
    for policy in ("lru", "protected_lru"):
        for pf in (0, 6):
            log(f"case policy={policy} prefetch_slots={pf}")
            runs[(policy, pf)] = _run(policy, pf, pool)
            s = runs[(policy, pf)][1]
            log(f"policy={policy} prefetch={pf}: fills={s['fills']} hits={s['hits']} misses={s['misses']} "
                f"prefetch_fills={s['prefetch_fills']} prefetch_used={s['prefetch_used']} "
                f"evictions={s['evictions']}")
    ref = runs[("lru", 0)][0]
    for k, (outs, s) in runs.items():
        assert outs == ref, k
        assert s["fills_in_flight"] == 0 and s["consumers_live"] == 0
        if k[1]:
            assert s["prefetch_fills"] > 0 and 0 < s["prefetch_used"] <= s["prefetch_fills"], s
        else:
            assert s["prefetch_fills"] == 0
