"""Seeded synthetic inputs for the slot-backed MoE layer.

This module is shared by the HIP path's tests/bench and by the CPU oracle's
tests.  It holds none of the layer's arithmetic: it only draws random numbers
and stores them in the byte formats the layer consumes (fp32, bf16, and a
symmetric 4-bit block format).  Every draw comes from numpy's PCG64 seeded by a
SeedSequence over (MASTER, workload, layer, kind, index, step), so any object
can be regenerated alone.

Byte formats (little endian):

* ``f32``   -- IEEE binary32.
* ``bf16``  -- the upper 16 bits of binary32 after round-to-nearest-even.
* ``q4b32`` -- a matrix [rows, cols] is stored as nibbles [rows, cols/2]
  (element 2j in the low nibble of byte j, 2j+1 in the high nibble, 4-bit
  two's complement, range [-8, 7]) followed by fp16 scales [rows, cols/32]
  (one per 32 consecutive elements of a row).  Value = scale * q.  The
  quantizer below only builds test data: scale = fp16(amax / 7),
  q = clamp(rint(w / scale), -8, 7), amax == 0 gives scale 0 and q 0.

* ``kq``    -- a mix of two super-block formats with 256-element super-blocks
  along each row (cols % 256 == 0), stored planar:
  ``k4`` (4.5 bits per weight, for Wg and Wu): nibbles [rows, cols/2] (element
  2j in the low nibble of byte j, unsigned 0..15), then one 16-byte header per
  row and super-block: fp16 d, fp16 dmin, eight 6-bit sub-block scales (48
  bits, little endian, scale j at bits 6j..6j+5), eight 6-bit sub-block mins
  likewise; value = d * sc_j * q - dmin * m_j for the j-th 32-element
  sub-block.  ``k6`` (6.5625 bits per weight, for Wd): low nibbles
  [rows, cols/2] (as above), high 2-bit parts [rows, cols/4] (element 4j + t
  at bits 2t..2t+1 of byte j), int8 scales [rows, cols/16] (one per 16
  elements), fp16 d [rows, cols/256]; q = low | high << 4 in 0..63 and value
  = d * sc_j * (q - 32).  The quantizers below only build test data.

An expert object is the concatenation [Wg | Wu | Wd] with Wg, Wu of shape
[I, d] (row-major, the reduction axis d contiguous) and Wd of shape [d, I]
(reduction axis I contiguous).  The router weight is stored [E, d].

Workload shapes follow the paper's model (48 MoE layers of 512 experts,
Implementation, and "Output-Exact Execution Beyond the Full-Residency
Envelope"); expert popularity priors (Dirichlet, Zipf) and
the bias temperature are this build's recipe for "every expert receives
tokens, with uneven counts".
"""
from __future__ import annotations

import os
import dataclasses
from typing import Optional

import numpy as np

MASTER = 20260821

# kinds used in the seed tuple
KIND_X = 0
KIND_ROUTER = 1
KIND_PRIOR = 2
KIND_EXPERT = 3
KIND_SHARED = 4
KIND_PERM = 5

WDTYPES = ("f32", "bf16", "q4b32", "kq")


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """Shape of one routed-expert layer.  ``T`` tokens, hidden ``d``, ``E``
    routed experts, top-``K``, expert intermediate ``I`` (shared expert uses
    the same ``I``)."""

    T: int
    d: int
    E: int
    K: int
    I: int
    wdtype: str = "bf16"
    shared: bool = True

    def __post_init__(self):
        assert self.wdtype in WDTYPES, self.wdtype
        assert 1 <= self.K <= self.E

    @property
    def xdtype(self) -> str:
        """Storage type of hidden states and router weight."""
        return "f32" if self.wdtype == "f32" else "bf16"

    def object_bytes(self) -> int:
        return object_nbytes(self.d, self.I, self.wdtype)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One named synthetic workload."""

    name: str
    wid: int                      # workload id in the seed tuple
    shape: LayerShape
    prior: str = "none"           # none | dirichlet | zipf
    prior_param: float = 0.0      # Dirichlet alpha or Zipf exponent
    tau: float = 0.0              # bias = tau * ln(p)
    n_layers: int = 1
    capacity: int = 64            # slots per layer for the LRU arm


WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", 1, LayerShape(64, 256, 16, 2, 128, "f32"),
                         capacity=4),
    "decode_bf16": Workload("decode_bf16", 2, LayerShape(16, 2048, 512, 10, 512, "bf16"),
                            capacity=64),
    "prefill_bf16": Workload("prefill_bf16", 3, LayerShape(32768, 2048, 512, 10, 512, "bf16"),
                             prior="dirichlet", prior_param=0.3, tau=0.2, capacity=512),
    "stack_bf16": Workload("stack_bf16", 4, LayerShape(4096, 2048, 512, 10, 512, "bf16"),
                           prior="zipf", prior_param=1.1, tau=0.3, n_layers=48, capacity=64),
    "prefill_q4": Workload("prefill_q4", 5, LayerShape(32768, 2048, 512, 10, 512, "q4b32"),
                           prior="zipf", prior_param=1.5, tau=0.3, capacity=512),
    "decode_q4": Workload("decode_q4", 5, LayerShape(1, 2048, 512, 10, 512, "q4b32"),
                          prior="zipf", prior_param=1.5, tau=0.3, capacity=512),
    # the quantized-expert mix (Wg, Wu 4.5 bits per weight, Wd 6.5625)
    "prefill_kq": Workload("prefill_kq", 6, LayerShape(32768, 2048, 512, 10, 512, "kq"),
                           prior="zipf", prior_param=1.5, tau=0.3, capacity=512),
    "decode_kq": Workload("decode_kq", 6, LayerShape(16, 2048, 512, 10, 512, "kq"),
                          prior="zipf", prior_param=1.5, tau=0.3, capacity=512),
}


def rng(wid: int, layer: int, kind: int, index: int = 0, step: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        [MASTER, int(wid), int(layer), int(kind), int(index), int(step)])))


# ----------------------------------------------------------------------------
# storage conversions (data construction only)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round binary32 to bfloat16 (nearest, ties to even); finite input."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    assert np.all((u & 0x7F800000) != 0x7F800000), "non-finite input"
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def quantize_q4b32(w: np.ndarray) -> bytes:
    """Quantize a float32 matrix [rows, cols] (cols % 32 == 0) to the q4b32
    byte layout described in the module docstring."""
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    assert cols % 32 == 0
    blk = w.reshape(rows, cols // 32, 32)
    amax = np.abs(blk).max(axis=2)
    scale16 = (amax / np.float32(7.0)).astype(np.float16)
    s32 = scale16.astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(s32[:, :, None] > 0, np.rint(blk / s32[:, :, None]), 0.0)
    q = np.clip(q, -8, 7).astype(np.int8).reshape(rows, cols)
    nib = (q.astype(np.uint8) & np.uint8(0x0F))
    packed = (nib[:, 0::2] | (nib[:, 1::2] << np.uint8(4))).astype(np.uint8)
    return packed.tobytes() + scale16.view(np.uint16).tobytes()


def q4b32_matrix_nbytes(rows: int, cols: int) -> int:
    return rows * cols // 2 + rows * (cols // 32) * 2


def k4_matrix_nbytes(rows: int, cols: int) -> int:
    return rows * cols // 2 + rows * (cols // 256) * 16


def k6_matrix_nbytes(rows: int, cols: int) -> int:
    return rows * cols // 2 + rows * cols // 4 + rows * cols // 16 + rows * (cols // 256) * 2


def _pack6(v):
    """Eight 6-bit values per row of v [n, 8] -> [n, 6] bytes, value j at bits 6j.. (little endian)."""
    import numpy as np
    v = np.asarray(v, dtype=np.uint64)
    word = np.zeros(v.shape[0], dtype=np.uint64)
    for j in range(8):
        word |= (v[:, j] & np.uint64(63)) << np.uint64(6 * j)
    return np.stack([((word >> np.uint64(8 * b)) & np.uint64(255)).astype(np.uint8) for b in range(6)], axis=1)


def _fp16_at_least(v: np.ndarray) -> np.ndarray:
    """The fp16 nearest to v, moved up one step where it fell below v."""
    h = np.asarray(v, dtype=np.float64).astype(np.float16)
    low = h.astype(np.float64) < v
    h[low] = np.nextafter(h[low], np.float16(np.inf))
    return h


def quantize_k4(w: np.ndarray) -> bytes:
    """w [rows, cols] (cols % 256 == 0) -> the k4 layout.  Per 32-element
    sub-block: lo = min(0, min w), hi = max(0, max w), a = (hi - lo) / 15,
    b = -lo; per super-block d = max a / 63 and dmin = max b / 63 in fp16
    (rounded up), sc = ceil(a / d), m = ceil(b / dmin) in 0..63 (so the step
    d sc covers a and the offset dmin m covers b), q = clamp(rint((w + dmin m)
    / (d sc)), 0, 15) (0 where d sc = 0)."""
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    assert cols % 256 == 0
    nsb = cols // 256
    sub = w.reshape(rows, nsb, 8, 32).astype(np.float64)
    lo = np.minimum(sub.min(axis=3), 0.0)
    hi = np.maximum(sub.max(axis=3), 0.0)
    a, b = (hi - lo) / 15.0, -lo
    d16 = _fp16_at_least(a.max(axis=2) / 63.0)
    m16 = _fp16_at_least(b.max(axis=2) / 63.0)
    d, dm = d16.astype(np.float64), m16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        sc = np.where(d[..., None] > 0, np.ceil(a / d[..., None]), 0.0).clip(0, 63)
        mn = np.where(dm[..., None] > 0, np.ceil(b / dm[..., None]), 0.0).clip(0, 63)
        step = d[..., None] * sc
        q = np.where(step[..., None] > 0, np.rint((sub + (dm[..., None] * mn)[..., None]) / step[..., None]), 0.0)
    q = q.clip(0, 15).astype(np.uint8).reshape(rows, cols)
    nib = (q[:, 0::2] | (q[:, 1::2] << np.uint8(4))).astype(np.uint8)
    hdr = np.zeros((rows, nsb, 16), dtype=np.uint8)
    hdr[:, :, 0:2] = d16.view(np.uint8).reshape(rows, nsb, 2)
    hdr[:, :, 2:4] = m16.view(np.uint8).reshape(rows, nsb, 2)
    hdr[:, :, 4:10] = _pack6(sc.reshape(-1, 8).astype(np.int64)).reshape(rows, nsb, 6)
    hdr[:, :, 10:16] = _pack6(mn.reshape(-1, 8).astype(np.int64)).reshape(rows, nsb, 6)
    return nib.tobytes() + hdr.tobytes()


def quantize_k6(w: np.ndarray) -> bytes:
    """w [rows, cols] (cols % 256 == 0) -> the k6 layout.  Per 16-element
    sub-block s = amax / 31; per super-block d = max s / 127 in fp16 (rounded
    up), sc = ceil(s / d) in 0..127 (the step d sc covers s), q =
    clamp(rint(w / (d sc)) + 32, 0, 63) (32 where d sc = 0)."""
    w = np.asarray(w, dtype=np.float32)
    rows, cols = w.shape
    assert cols % 256 == 0
    nsb = cols // 256
    sub = w.reshape(rows, nsb, 16, 16).astype(np.float64)
    s = np.abs(sub).max(axis=3) / 31.0
    d16 = _fp16_at_least(s.max(axis=2) / 127.0)
    d = d16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        sc = np.where(d[..., None] > 0, np.ceil(s / d[..., None]), 0.0).clip(-128, 127)
        step = d[..., None] * sc
        q = np.where(step[..., None] != 0, np.rint(sub / step[..., None]) + 32, 32.0)
    q = q.clip(0, 63).astype(np.uint8).reshape(rows, cols)
    low = q & np.uint8(15)
    ql = (low[:, 0::2] | (low[:, 1::2] << np.uint8(4))).astype(np.uint8)
    hi2 = (q >> np.uint8(4)) & np.uint8(3)
    qh = (hi2[:, 0::4] | (hi2[:, 1::4] << np.uint8(2)) | (hi2[:, 2::4] << np.uint8(4)) |
          (hi2[:, 3::4] << np.uint8(6))).astype(np.uint8)
    return ql.tobytes() + qh.tobytes() + sc.astype(np.int8).tobytes() + d16.tobytes()


def object_nbytes(d: int, I: int, wdtype: str) -> int:
    if wdtype == "f32":
        return 3 * I * d * 4
    if wdtype == "bf16":
        return 3 * I * d * 2
    if wdtype == "kq":
        return 2 * k4_matrix_nbytes(I, d) + k6_matrix_nbytes(d, I)
    return 2 * q4b32_matrix_nbytes(I, d) + q4b32_matrix_nbytes(d, I)


def encode_matrix(w: np.ndarray, wdtype: str) -> bytes:
    if wdtype == "f32":
        return np.ascontiguousarray(w, dtype=np.float32).tobytes()
    if wdtype == "bf16":
        return f32_to_bf16_bits(w).tobytes()
    if wdtype in ("k4", "k6"):
        return quantize_k4(w) if wdtype == "k4" else quantize_k6(w)
    return quantize_q4b32(w)


def encode_dense(a: np.ndarray, dtype: str) -> np.ndarray:
    """Hidden states / router weight storage: f32 or bf16 (as uint16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(a, dtype=np.float32)
    return f32_to_bf16_bits(a)


# ----------------------------------------------------------------------------
# draws
# ----------------------------------------------------------------------------

def expert_object(wl: Workload, layer: int, expert: int, shared: bool = False) -> np.ndarray:
    """One expert object [Wg | Wu | Wd] as a uint8 array.  ``shared`` selects
    the layer's always-on shared expert (its own seed stream)."""
    s = wl.shape
    g = rng(wl.wid, layer, KIND_SHARED if shared else KIND_EXPERT, expert)
    wg = g.standard_normal((s.I, s.d), dtype=np.float32) * np.float32(0.02)
    wu = g.standard_normal((s.I, s.d), dtype=np.float32) * np.float32(0.02)
    wd = g.standard_normal((s.d, s.I), dtype=np.float32) * np.float32(0.02)
    if s.wdtype == "kq":       # gate / up in the 4.5-bit format, down in the 6.5625-bit one
        b = encode_matrix(wg, "k4") + encode_matrix(wu, "k4") + encode_matrix(wd, "k6")
    else:
        b = encode_matrix(wg, s.wdtype) + encode_matrix(wu, s.wdtype) + encode_matrix(wd, s.wdtype)
    out = np.frombuffer(b, dtype=np.uint8).copy()
    assert out.nbytes == s.object_bytes()
    return out


def hidden_states(wl: Workload, layer: int = 0, step: int = 0, T: Optional[int] = None) -> np.ndarray:
    """x [T, d]: float32 array (f32 workloads) or uint16 bf16 bits."""
    s = wl.shape
    T = s.T if T is None else T
    g = rng(wl.wid, layer, KIND_X, 0, step)
    return encode_dense(g.standard_normal((T, s.d), dtype=np.float32), s.xdtype)


def router_weight(wl: Workload, layer: int = 0) -> np.ndarray:
    """Wr stored [E, d]: float32 (f32 workloads) or uint16 bf16 bits."""
    s = wl.shape
    g = rng(wl.wid, layer, KIND_ROUTER)
    return encode_dense(g.standard_normal((s.E, s.d), dtype=np.float32) * np.float32(0.02), s.xdtype)


def stack_expert_map(wl: Workload, layer: int) -> np.ndarray:
    """Layer stacks draw their routed-expert objects from one pool of E
    distinct seeded objects (pool object i = ``expert_object(wl, 0, i)``):
    expert e of layer l is pool object map[e], with map a seeded permutation
    per layer.  Host windows then hold E objects instead of n_layers * E."""
    if layer == 0:
        return np.arange(wl.shape.E)
    return rng(wl.wid, layer, KIND_PERM, 1).permutation(wl.shape.E)


def popularity_prior(wl: Workload, layer: int = 0) -> Optional[np.ndarray]:
    """Per-expert popularity p (sums to 1) or None for the unbiased workloads."""
    E = wl.shape.E
    if wl.prior == "none":
        return None
    g = rng(wl.wid, layer, KIND_PRIOR)
    if wl.prior == "dirichlet":
        p = g.dirichlet(np.full(E, wl.prior_param))
    elif wl.prior == "zipf":
        ranks = np.arange(1, E + 1, dtype=np.float64) ** (-wl.prior_param)
        perm = rng(wl.wid, layer, KIND_PERM).permutation(E)
        p = np.empty(E)
        p[perm] = ranks / ranks.sum()
    else:
        raise ValueError(wl.prior)
    return np.maximum(p, 1e-30)


def router_bias(wl: Workload, layer: int = 0) -> Optional[np.ndarray]:
    """bias [E] float32 = tau * ln p, or None."""
    p = popularity_prior(wl, layer)
    if p is None:
        return None
    return (wl.tau * np.log(p)).astype(np.float32)


@dataclasses.dataclass
class LayerInputs:
    wl: Workload
    layer: int
    x: np.ndarray                   # [T, d] f32 or bf16 bits
    wr: np.ndarray                  # [E, d] f32 or bf16 bits
    bias: Optional[np.ndarray]      # [E] f32 or None
    experts: list                   # E uint8 objects (or None when lazy)
    shared: Optional[np.ndarray]    # uint8 object

    def expert(self, e: int) -> np.ndarray:
        if self.experts[e] is None:
            self.experts[e] = expert_object(self.wl, self.layer, e)
        return self.experts[e]

    def prefetch(self, ids=None, threads: int = 0) -> "LayerInputs":
        """Draw the listed expert objects (default all) on a thread pool."""
        import concurrent.futures
        import os
        ids = range(len(self.experts)) if ids is None else ids
        todo = [e for e in ids if self.experts[e] is None]
        n = threads or min(16, os.cpu_count() or 1)
        with concurrent.futures.ThreadPoolExecutor(n) as ex:
            for e, obj in zip(todo, ex.map(lambda e: expert_object(self.wl, self.layer, e), todo)):
                self.experts[e] = obj
        return self


def layer_inputs(wl: Workload, layer: int = 0, step: int = 0, T: Optional[int] = None,
                 lazy: bool = False, shape: Optional[LayerShape] = None) -> LayerInputs:
    """All inputs of one layer.  ``lazy`` defers drawing expert objects until
    ``LayerInputs.expert(e)`` is called.  ``shape`` overrides the workload's
    shape (same seeds) for reduced test sizes."""
    if shape is not None:
        wl = dataclasses.replace(wl, shape=shape)
    s = wl.shape
    li = LayerInputs(
        wl=wl, layer=layer,
        x=hidden_states(wl, layer, step, T),
        wr=router_weight(wl, layer),
        bias=router_bias(wl, layer),
        experts=[None] * s.E,
        shared=expert_object(wl, layer, 0, shared=True) if s.shared else None,
    )
    return li if lazy else li.prefetch()


# ----------------------------------------------------------------------------
# canonical files (storage layout only)
# ----------------------------------------------------------------------------

def component_sizes(shape: LayerShape):
    """Byte sizes of an expert object's components [Wg, Wu, Wd]."""
    if shape.wdtype == "kq":
        return [k4_matrix_nbytes(shape.I, shape.d), k4_matrix_nbytes(shape.I, shape.d),
                k6_matrix_nbytes(shape.d, shape.I)]
    if shape.wdtype == "f32":
        m = lambda r, c: r * c * 4  # noqa: E731
    elif shape.wdtype == "bf16":
        m = lambda r, c: r * c * 2  # noqa: E731
    else:
        m = q4b32_matrix_nbytes
    return [m(shape.I, shape.d), m(shape.I, shape.d), m(shape.d, shape.I)]


def write_canonical_file(path: str, objects, comp_sizes, seed: int = 0, gap: int = 1000, sync: bool = False):
    """Write objects (uint8 arrays, each the concatenation of its components)
    to one canonical file with every component at its own offset: components
    in a seeded shuffled order, each followed by ``gap`` filler bytes so that
    no extent is aligned to the direct-I/O block (``sync``: flushed to the
    device before returning).  Returns the extents as (object index,
    component, offset, nbytes) tuples; the same arguments give the same file."""
    import numpy as np
    order = [(i, c) for i in range(len(objects)) for c in range(len(comp_sizes))]
    perm = np.random.Generator(np.random.PCG64(np.random.SeedSequence([MASTER, 900, seed]))).permutation(len(order))
    starts = [0]
    for c in comp_sizes[:-1]:
        starts.append(starts[-1] + c)
    extents, off = [], 0
    with open(path, "wb") as fh:
        for j in perm:
            i, c = order[j]
            obj = np.asarray(objects[i], dtype=np.uint8)
            fh.write(obj[starts[c]:starts[c] + comp_sizes[c]].tobytes())
            extents.append((i, c, off, comp_sizes[c]))
            off += comp_sizes[c]
            fh.write(b"\xa5" * gap)
            off += gap
        if sync:
            fh.flush()
            os.fsync(fh.fileno())
    return sorted(extents)
