"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with the pinned fact.  ``tests/test_oracle_pins.py`` runs
them on the clean build; ``tests/test_oracle_mutants.py`` runs them on builds
with one planted mistake each and requires that some pin fails.

Sources of truth used here (none of them is the oracle's own code):
* IEEE 754 binary16 / bfloat16 bit patterns (golden text fixtures);
* a hand-decoded 4-bit block (golden fixture);
* exact rational arithmetic (``fractions.Fraction``) for brute-force top-K;
* numpy / scipy library routines for special cases that reduce to them
  (matrix products, ``scipy.special.softmax`` / ``expit``);
* closed forms and invariants (zero input, power-of-two scaling, relabeling,
  restricted softmax ratios, weights summing to one, unit mean square after
  the stack's input normalisation).
"""
from __future__ import annotations

import itertools
import os
from fractions import Fraction

import numpy as np
import scipy.special

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TINY = synth.WORKLOADS["tiny_f32"]          # T=64 d=256 E=16 K=2 I=128 fp32
SMALL_BF16 = synth.LayerShape(12, 64, 8, 3, 32, "bf16")
SMALL_Q4 = synth.LayerShape(6, 64, 6, 2, 64, "q4b32")
SMALL_KQ = synth.LayerShape(5, 256, 6, 2, 256, "kq")


def _tiny_inputs(shape=None, wl=TINY, bias=False):
    li = synth.layer_inputs(wl, shape=shape)
    if bias:
        g = synth.rng(99, 0, 7)
        li.bias = (g.standard_normal(li.wr.shape[0]) * 0.3).astype(np.float32)
    return li


def _dense(o, arr, dtype, rows, cols):
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float64).reshape(rows, cols)
    return o.dequant(dtype, rows, cols, arr)


# ---------------------------------------------------------------- formats

def pin_formats(o):
    with open(os.path.join(GOLDEN, "fp_formats.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            fmt, bits, val = line.split()
            got = o.fp16_to_f64(int(bits, 16)) if fmt == "fp16" else o.bf16_to_f64(int(bits, 16))
            want = float(val)
            assert got == want and np.signbit(got) == np.signbit(want), (fmt, bits, got, want)


def pin_bf16_rounding(o):
    with open(os.path.join(GOLDEN, "bf16_rounding.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            expr, bits = line.rsplit(None, 1)
            v = eval(expr, {"__builtins__": {}})   # fixture arithmetic on literals only
            assert o.f64_to_bf16(v) == int(bits, 16), (expr, hex(o.f64_to_bf16(v)), bits)
    # agreement with the independent float32 route on random binary32 values
    g = np.random.default_rng(5)
    a = (g.standard_normal(2000) * 10.0 ** g.integers(-30, 30, 2000)).astype(np.float32)
    want = synth.f32_to_bf16_bits(a)
    got = o.f64_to_bf16_array(a.astype(np.float64))
    assert np.array_equal(got, want)


def pin_q4_block(o):
    rows = {}
    with open(os.path.join(GOLDEN, "q4b32_block.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            k, *vals = line.split()
            rows[k] = vals
    raw = bytes(int(b, 16) for b in rows["bytes"]) + int(rows["scale"][0], 16).to_bytes(2, "little")
    q = np.array([int(v) for v in rows["q"]], dtype=np.float64)
    got = o.dequant("q4b32", 1, 32, np.frombuffer(raw, dtype=np.uint8))
    assert np.array_equal(got[0], 0.5 * q), (got, q)


def pin_q4_quantizer_bound(o):
    """Dequantised values lie within half a quantum of the source (plus the
    fp16 rounding of the scale), block by block."""
    g = np.random.default_rng(11)
    w = (g.standard_normal((8, 128)) * 0.02).astype(np.float32)
    w[3, 32:64] = 0.0                                   # all-zero block: scale 0
    raw = np.frombuffer(synth.quantize_q4b32(w), dtype=np.uint8)
    deq = o.dequant("q4b32", 8, 128, raw)
    blk = np.abs(w.astype(np.float64)).reshape(8, 4, 32).max(axis=2)
    s = blk / 7.0
    bound = np.repeat(s * 0.5 + blk * 2.0 ** -10, 32, axis=1)
    assert np.all(np.abs(deq - w) <= bound + 1e-12)
    assert np.all(deq[3, 32:64] == 0.0)


def _k4_block_bytes():
    """The k4 super-block of the golden fixture, packed from the format
    definition with plain integer arithmetic."""
    nib = bytes((((2 * i) % 16) | (((2 * i + 1) % 16) << 4)) for i in range(128))
    sc = sum((j + 1) << (6 * j) for j in range(8))
    mn = sum(j << (6 * j) for j in range(8))
    hdr = (0x3800).to_bytes(2, "little") + (0x3400).to_bytes(2, "little") + sc.to_bytes(6, "little") + \
        mn.to_bytes(6, "little")
    return nib + hdr


def _k6_block_bytes():
    q = [(5 * k) % 64 for k in range(256)]
    ql = bytes(((q[2 * i] & 15) | ((q[2 * i + 1] & 15) << 4)) for i in range(128))
    qh = bytes(sum(((q[4 * i + t] >> 4) & 3) << (2 * t) for t in range(4)) for i in range(64))
    sc = bytes(((j - 8) & 0xFF) for j in range(16))
    return ql + qh + sc + (0x3000).to_bytes(2, "little")


def pin_kquant_blocks(o):
    """Hand-derived elements of one super-block of each quantized-expert format."""
    want = {"k4": {}, "k6": {}}
    with open(os.path.join(GOLDEN, "kquant_blocks.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                fmt, k, v = line.split()
                want[fmt][int(k)] = float(v)
    for fmt, raw in (("k4", _k4_block_bytes()), ("k6", _k6_block_bytes())):
        assert len(raw) == o.matrix_nbytes(fmt, 1, 256)
        got = o.dequant(fmt, 1, 256, np.frombuffer(raw, dtype=np.uint8))[0]
        for k, v in want[fmt].items():
            assert got[k] == v, (fmt, k, got[k], v)


def pin_kquant_quantizer_bound(o):
    """The test-data quantizers' outputs decode within the formats' error
    bounds: k4 within half a step (the step d*sc is below a + d) plus the
    offset's excess (below dmin); k6 within half a step (below (s + d) / 2,
    s = amax / 31); an all-zero super-block decodes to zeros."""
    g = np.random.default_rng(12)
    w = (g.standard_normal((6, 512)) * 0.02).astype(np.float32)
    w[2, 256:] = 0.0                                   # an all-zero super-block
    dq = o.dequant("k4", 6, 512, np.frombuffer(synth.quantize_k4(w), dtype=np.uint8))
    sub = w.astype(np.float64).reshape(6, 2, 8, 32)
    a = (np.maximum(sub.max(axis=3), 0) - np.minimum(sub.min(axis=3), 0)) / 15.0
    d = a.max(axis=2, keepdims=True) / 63.0
    b = -np.minimum(sub.min(axis=3), 0)
    dm = b.max(axis=2, keepdims=True) / 63.0
    bound = (0.5 * (a + d) + dm) * (1 + 2.0 ** -9) + 1e-9
    assert np.all(np.abs(dq - w).reshape(6, 2, 8, 32) <= bound[..., None])
    assert np.all(dq[2, 256:] == 0.0)
    dq6 = o.dequant("k6", 6, 512, np.frombuffer(synth.quantize_k6(w), dtype=np.uint8))
    sub6 = w.astype(np.float64).reshape(6, 2, 16, 16)
    s6 = np.abs(sub6).max(axis=3) / 31.0
    d6 = s6.max(axis=2, keepdims=True) / 127.0
    bound6 = (0.5 * (s6 + d6)) * (1 + 2.0 ** -9) + 1e-9
    assert np.all(np.abs(dq6 - w).reshape(6, 2, 16, 16) <= bound6[..., None])
    assert np.all(dq6[2, 256:] == 0.0)


# ---------------------------------------------------------------- router

def pin_router_matches_matmul(o):
    for shape, bias in ((TINY.shape, True), (SMALL_BF16, True)):
        li = _tiny_inputs(shape, bias=bias)
        s = shape
        x = _dense(o, li.x, s.xdtype, s.T, s.d)
        wr = _dense(o, li.wr, s.xdtype, s.E, s.d)
        L = o.router_logits(li.x, li.wr, li.bias, s.xdtype)
        ref = x @ wr.T + li.bias.astype(np.float64)[None, :]
        assert np.allclose(L, ref, rtol=0, atol=1e-12 * max(1.0, np.abs(ref).max()))


def pin_topk_bruteforce(o):
    """Exhaustive search over all K-subsets: maximise the exact sum of logits,
    ties broken by the lexicographically smallest sorted id tuple.  Includes
    rows with deliberate exact ties."""
    g = np.random.default_rng(3)
    E, K = 7, 3
    L = g.standard_normal((40, E))
    L[:10] = np.round(L[:10] * 2) / 2           # many exact ties
    L[10] = 0.0                                  # all tied
    L[11, [1, 4, 6]] = 5.0
    L[11, [0, 2, 3, 5]] = 5.0                    # seven-way tie at the top
    idx, gap = o.select_topk(L, K)
    for t in range(L.shape[0]):
        best, best_key = None, None
        for sub in itertools.combinations(range(E), K):
            key = (-sum(Fraction(float(L[t, e])) for e in sub), sub)
            if best_key is None or key < best_key:
                best, best_key = sub, key
        assert tuple(idx[t]) == best, (t, idx[t], best)
        srt = sorted(L[t], reverse=True)
        assert gap[t] == srt[K - 1] - srt[K]
    assert tuple(idx[10]) == (0, 1, 2)


def pin_topk_zero_router(o):
    """Wr = 0 and b = 0: every logit ties, so S = {0..K-1} and w = 1/K."""
    s = TINY.shape
    x = synth.hidden_states(TINY)
    wr = np.zeros((s.E, s.d), dtype=np.float32)
    li = _tiny_inputs()
    r = o.moe_layer(x, wr, None, li.experts, li.shared, s.K, s.I, "f32", "f32", tokens=range(4))
    assert np.all(r["idx"] == np.arange(s.K))
    assert np.all(r["w"] == 1.0 / s.K)


def pin_gate_weights(o):
    g = np.random.default_rng(4)
    L = g.standard_normal((30, 9)) * 3
    # K = E: the restricted softmax is the full softmax (library routine)
    idx = np.tile(np.arange(9, dtype=np.int32), (30, 1))
    w = o.gate_weights(L, idx)
    assert np.allclose(w, scipy.special.softmax(L, axis=1), rtol=1e-13, atol=0)
    # K < E: sums to one, ratios are exp of logit differences
    idx, _ = o.select_topk(L, 4)
    w = o.gate_weights(L, idx)
    assert np.all(np.abs(w.sum(axis=1) - 1.0) <= 1e-12)
    sel = np.take_along_axis(L, idx.astype(np.int64), axis=1)
    assert np.allclose(w[:, 1:] / w[:, :1], np.exp(sel[:, 1:] - sel[:, :1]), rtol=1e-12)


# ---------------------------------------------------------------- permutation

def pin_permutation(o):
    g = np.random.default_rng(6)
    T, E, K = 50, 12, 4
    idx = np.sort(np.stack([g.choice(E, K, replace=False) for _ in range(T)]), axis=1).astype(np.int32)
    counts, offsets, perm, inv = o.permute(idx, E)
    assert np.array_equal(counts, np.bincount(idx.ravel(), minlength=E))
    assert offsets[0] == 0 and np.array_equal(np.diff(offsets), counts)
    # rows ordered by (expert, token): numpy's stable sort of the keys
    keys = idx.astype(np.int64) * T + np.arange(T)[:, None]
    order = np.argsort(keys.ravel(), kind="stable")
    assert np.array_equal(perm, order // K)
    assert np.array_equal(inv.ravel()[order], np.arange(T * K))
    # brute force on a tiny case: walk experts then tokens
    rows = [(e, t) for e in range(E) for t in range(T) if e in idx[t]]
    assert [perm[r] for r in range(len(rows))] == [t for _, t in rows]


# ---------------------------------------------------------------- experts / layer

def pin_expert_ffn_special(o):
    """d = I with Wg = diag(a), Wu = I, Wd = I: y_i = x_i * sigmoid(a_i x_i) * a_i x_i
    reduces to scipy's expit; x = 0 gives 0 exactly; Wd and Wu scale linearly."""
    n = 32
    a = np.linspace(-3, 3, n).astype(np.float32)
    wg = np.diag(a).astype(np.float32)
    eye = np.eye(n, dtype=np.float32)
    obj = np.frombuffer(wg.tobytes() + eye.tobytes() + eye.tobytes(), dtype=np.uint8)
    x = np.linspace(-2, 2, n)
    y = o.expert_ffn(obj, x, n, n, "f32")
    z = a.astype(np.float64) * x
    assert np.allclose(y, z * scipy.special.expit(z) * x, rtol=1e-14, atol=1e-300)
    assert np.all(o.expert_ffn(obj, np.zeros(n), n, n, "f32") == 0.0)
    li = _tiny_inputs()
    s = TINY.shape
    obj = li.experts[3]
    xt = np.asarray(li.x[5], dtype=np.float64)
    y1 = o.expert_ffn(obj, xt, s.d, s.I, "f32")
    wg_, wu_, wd_ = [m.astype(np.float32) for m in o.expert_matrices(obj, s.d, s.I, "f32")]
    obj2 = np.frombuffer(wg_.tobytes() + wu_.tobytes() + (2 * wd_).tobytes(), dtype=np.uint8)
    assert np.array_equal(o.expert_ffn(obj2, xt, s.d, s.I, "f32"), 2 * y1)
    obj3 = np.frombuffer(wg_.tobytes() + (4 * wu_).tobytes() + wd_.tobytes(), dtype=np.uint8)
    assert np.array_equal(o.expert_ffn(obj3, xt, s.d, s.I, "f32"), 4 * y1)


def pin_expert_ffn_matmul(o):
    """Cross-check of the gated-SiLU FFN against numpy matrix products with
    scipy's expit, in all three storage formats."""
    for shape, wl in ((TINY.shape, TINY), (SMALL_BF16, TINY), (SMALL_Q4, TINY), (SMALL_KQ, TINY)):
        li = _tiny_inputs(shape)
        s = shape
        x = _dense(o, li.x, s.xdtype, s.T, s.d)
        for e in (0, s.E - 1):
            wg, wu, wd = o.expert_matrices(li.experts[e], s.d, s.I, s.wdtype)
            for t in (0, s.T - 1):
                g, u = wg @ x[t], wu @ x[t]
                ref = wd @ (g * scipy.special.expit(g) * u)
                y = o.expert_ffn(li.experts[e], x[t], s.d, s.I, s.wdtype)
                assert np.allclose(y, ref, rtol=1e-12, atol=1e-14 * np.abs(ref).max())


def _dense_layer(o, li, shape):
    """All-expert masked evaluation (a different loop order from the oracle's
    sparse per-token walk): out = shared + sum_e mask[t,e] w[t,e] FFN_e(x_t)."""
    s = shape
    x = _dense(o, li.x, s.xdtype, s.T, s.d)
    L = o.router_logits(li.x, li.wr, li.bias, s.xdtype)
    idx, _ = o.select_topk(L, s.K)
    w = o.gate_weights(L, idx)
    W = np.zeros((s.T, s.E))
    np.put_along_axis(W, idx.astype(np.int64), w, axis=1)
    out = np.zeros((s.T, s.d))
    if li.shared is not None:
        wg, wu, wd = o.expert_matrices(li.shared, s.d, s.I, s.wdtype)
        g, u = x @ wg.T, x @ wu.T
        out += (g * scipy.special.expit(g) * u) @ wd.T
    for e in range(s.E):
        wg, wu, wd = o.expert_matrices(li.experts[e], s.d, s.I, s.wdtype)
        g, u = x @ wg.T, x @ wu.T
        out += W[:, e:e + 1] * ((g * scipy.special.expit(g) * u) @ wd.T)
    return out, idx, w


def pin_layer_dense(o):
    for shape, bias in ((TINY.shape, True), (SMALL_BF16, False), (SMALL_Q4, True), (SMALL_KQ, True)):
        li = _tiny_inputs(shape, bias=bias)
        s = shape
        ref, idx, w = _dense_layer(o, li, s)
        r = o.moe_layer(li.x, li.wr, li.bias, li.experts, li.shared, s.K, s.I, s.wdtype, s.xdtype)
        assert np.array_equal(r["idx"], idx)
        assert np.allclose(r["w"], w, rtol=1e-13, atol=0)
        err = np.abs(r["out"] - ref).max() / np.abs(ref).max()
        assert err <= 1e-12, err


def pin_layer_invariants(o):
    s = TINY.shape
    li = _tiny_inputs(bias=True)
    base = o.moe_layer(li.x, li.wr, li.bias, li.experts, li.shared, s.K, s.I, "f32", "f32")
    # x = 0: all logits equal the bias, every FFN is zero
    z = o.moe_layer(np.zeros_like(li.x), li.wr, li.bias, li.experts, li.shared, s.K, s.I, "f32", "f32")
    assert np.all(z["out"] == 0.0)
    # doubling every down projection doubles the output exactly
    def dbl(obj):
        m = [a.astype(np.float32) for a in o.expert_matrices(obj, s.d, s.I, "f32")]
        return np.frombuffer(m[0].tobytes() + m[1].tobytes() + (2 * m[2]).tobytes(), dtype=np.uint8)
    r2 = o.moe_layer(li.x, li.wr, li.bias, [dbl(e) for e in li.experts], dbl(li.shared),
                     s.K, s.I, "f32", "f32")
    assert np.array_equal(r2["out"], 2 * base["out"])
    # relabeling experts (objects, router rows and bias together) changes nothing
    p = synth.rng(1, 0, 9).permutation(s.E)
    wr = np.asarray(li.wr)[p]
    r3 = o.moe_layer(li.x, wr, li.bias[p], [li.experts[q] for q in p], li.shared,
                     s.K, s.I, "f32", "f32")
    assert np.array_equal(np.sort(p[r3["idx"]], axis=1), base["idx"])
    assert np.allclose(r3["out"], base["out"], rtol=0, atol=1e-12 * np.abs(base["out"]).max())
    # without the shared expert the output drops by exactly its FFN
    r4 = o.moe_layer(li.x, li.wr, li.bias, li.experts, None, s.K, s.I, "f32", "f32")
    for t in (0, 17):
        ys = o.expert_ffn(li.shared, np.asarray(li.x[t], np.float64), s.d, s.I, "f32")
        assert np.allclose(base["out"][t] - r4["out"][t], ys, rtol=0, atol=1e-12)
    # the bias moves selections: a huge bias on expert 5 puts it in every set
    b = li.bias.copy()
    b[5] = 1e3
    r5 = o.moe_layer(li.x, li.wr, b, li.experts, li.shared, s.K, s.I, "f32", "f32", tokens=range(8))
    assert np.all(np.any(r5["idx"] == 5, axis=1))
    # forced selection equal to the oracle's own gives the same output
    r6 = o.moe_layer(li.x, li.wr, li.bias, li.experts, li.shared, s.K, s.I, "f32", "f32",
                     forced_idx=base["idx"])
    assert np.array_equal(r6["out"], base["out"])


# ---------------------------------------------------------------- layer stack (residual stream)

def pin_residual_rows(o):
    """Hand-derived rows of the residual step (golden fixture)."""
    with open(os.path.join(GOLDEN, "residual_rows.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            hs, outs, want = (p.split() for p in line.split("|"))
            h = np.array([[float(v) for v in hs]])
            out = None if outs == ["-"] else np.array([[float(v) for v in outs]])
            hn, x = o.residual_step(h, out)
            assert [int(b, 16) for b in want] == x[0].tolist(), (line, [hex(v) for v in x[0]])
            assert np.array_equal(hn, h if out is None else h + out), line


def pin_residual_invariants(o):
    """Normalised rows have unit mean square (up to bf16 rounding); scaling a
    row by a power of two leaves x unchanged when the epsilon is negligible;
    the residual stream itself is the plain sum, exact in fp64."""
    g = np.random.default_rng(21)
    h = g.standard_normal((16, 512)) * 100.0
    out = g.standard_normal((16, 512)) * 30.0
    hn, x = o.residual_step(h, out)
    assert np.array_equal(hn, h + out)
    xv = synth.bf16_bits_to_f32(x).astype(np.float64)
    ms = (xv ** 2).mean(axis=1)
    assert np.all(np.abs(ms - 1.0) <= 2 * 2.0 ** -8), ms
    for k in (-4, 3, 10):
        _, xk = o.residual_step(h * 2.0 ** k, out * 2.0 ** k)
        assert np.array_equal(xk, x), k
    # each element is the nearest bf16 of h / rms: within half a bf16 step (2^-8 relative, plus the rms's
    # own relative error bound from fp64)
    ref = hn / np.sqrt((hn ** 2).mean(axis=1, keepdims=True))
    assert np.all(np.abs(xv - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-300)


def pin_stack_chain(o):
    """Two stacked layers equal their steps applied by hand: the second
    layer's input is the normalised sum of the first layer's input stream
    and output, and a layer with every routed and shared down projection zero
    leaves the residual stream unchanged."""
    s = SMALL_BF16
    li = _tiny_inputs(s, bias=True)
    ly = dict(wr=li.wr, bias=li.bias, experts=li.experts, shared=li.shared)
    h0 = synth.bf16_bits_to_f32(li.x).astype(np.float64) * 3.0
    r = o.stack(h0, [ly, ly], s.K, s.I, s.wdtype)
    x0 = o.f64_to_bf16_array(h0 / np.sqrt((h0 ** 2).mean(axis=1, keepdims=True) + 1e-6))
    assert np.array_equal(r["xs"][0], x0)
    out0 = o.moe_layer(x0, li.wr, li.bias, li.experts, li.shared, s.K, s.I, s.wdtype, "bf16")["out"]
    h1 = h0 + out0
    assert np.array_equal(r["xs"][1], o.f64_to_bf16_array(h1 / np.sqrt((h1 ** 2).mean(axis=1, keepdims=True)
                                                                         + 1e-6)))
    out1 = o.moe_layer(r["xs"][1], li.wr, li.bias, li.experts, li.shared, s.K, s.I, s.wdtype, "bf16")["out"]
    assert np.array_equal(r["h"], h1 + out1)
    nb = o.matrix_nbytes(s.wdtype, s.I, s.d)

    def no_down(obj):
        z = np.array(obj, dtype=np.uint8, copy=True)
        z[2 * nb:] = 0
        return z
    quiet = dict(wr=li.wr, bias=li.bias, experts=[no_down(e) for e in li.experts], shared=no_down(li.shared))
    rq = o.stack(h0, [quiet, quiet, quiet], s.K, s.I, s.wdtype)
    assert np.array_equal(rq["h"], h0) and np.array_equal(rq["xs"][2], x0)


ALL_PINS = [
    pin_formats, pin_bf16_rounding, pin_q4_block, pin_q4_quantizer_bound,
    pin_router_matches_matmul, pin_topk_bruteforce, pin_topk_zero_router, pin_gate_weights,
    pin_permutation, pin_expert_ffn_special, pin_expert_ffn_matmul, pin_layer_dense,
    pin_layer_invariants, pin_residual_rows, pin_residual_invariants, pin_stack_chain,
    pin_kquant_blocks, pin_kquant_quantizer_bound,
]
