"""Python binding of libmsi.so, the MI355X slot-backed MoE layer.

Argument marshalling only: every step of the layer runs in the HIP kernels of
``libmsi.so``; PyTorch provides device memory, pinned host windows and
streams.  The names mirror the C ABI in ``include/msi.h``.  Importing this
package fails loudly when the library has not been built (there is no
fallback).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmsi.so")

MSI_ABI_VERSION = 3
MSI_OK = 0
MSI_E_INVALID_ARG = -1
MSI_E_SHORT = -2
MSI_E_WRONG_OBJECT = -3
MSI_E_BUSY = -4
MSI_E_STALE = -5
MSI_E_DEVICE = -6
MSI_E_NOMEM = -7
MSI_E_STATE = -8
MSI_E_IO = -9
STATUS_NAMES = {0: "MSI_OK", -1: "MSI_E_INVALID_ARG", -2: "MSI_E_SHORT", -3: "MSI_E_WRONG_OBJECT",
                -4: "MSI_E_BUSY", -5: "MSI_E_STALE", -6: "MSI_E_DEVICE", -7: "MSI_E_NOMEM",
                -8: "MSI_E_STATE", -9: "MSI_E_IO"}
MSI_SOURCE_BUFFERED_OK = 1
FAULTS = {"short": 1, "eio": 2, "hold": 3}
POLICIES = {"lru": 0, "protected_lru": 1}

MSI_W_F32, MSI_W_BF16, MSI_W_Q4B32, MSI_W_KQ = 0, 1, 2, 3
MSI_NOALLOC_SCRATCH_BYTES = 64 << 20
WDTYPE = {"f32": MSI_W_F32, "bf16": MSI_W_BF16, "q4b32": MSI_W_Q4B32, "kq": MSI_W_KQ}
SLOT_STATES = {0: "Vacant", 1: "Loading", 2: "DeviceReady", 3: "InUse", 4: "Recyclable"}

_u32, _i32, _u64, _vp = ctypes.c_uint32, ctypes.c_int32, ctypes.c_uint64, ctypes.c_void_p


class msi_object_desc(ctypes.Structure):
    _fields_ = [("layer", _u32), ("expert", _u32), ("window", _u32), ("reserved", _u32),
                ("offset", _u64), ("nbytes", _u64)]


class msi_extent_desc(ctypes.Structure):
    _fields_ = [("layer", _u32), ("expert", _u32), ("component", _u32), ("file", _u32),
                ("offset", _u64), ("nbytes", _u64)]


class msi_source_desc(ctypes.Structure):
    _fields_ = [("files", ctypes.POINTER(ctypes.c_char_p)), ("n_files", _u32), ("inflight", _u32),
                ("flags", _u32), ("align", _u32), ("extents", ctypes.POINTER(msi_extent_desc)),
                ("n_extents", _u32), ("reserved", _u32)]


class msi_source_stats(ctypes.Structure):
    _fields_ = [(n, _u64) for n in ("reads_issued", "reads_completed", "reads_failed", "requests",
                                    "requests_ready", "requests_failed", "requests_stale", "logical_bytes",
                                    "physical_bytes", "padding_bytes", "peak_depth", "windows_busy")] + \
               [("read_seconds", ctypes.c_double), ("wait_seconds", ctypes.c_double),
                ("direct_files", _u32), ("buffered_files", _u32), ("bounced_reads", _u64)]


class msi_plan_desc(ctypes.Structure):
    _fields_ = [("abi_version", _u32), ("n_layers", _u32), ("n_experts", _u32), ("d_model", _u32),
                ("d_ff", _u32), ("top_k", _u32), ("wdtype", _u32), ("slots_per_layer", _u32),
                ("transient_slots", _u32), ("policy", _u32), ("slot_pool", _vp),
                ("slot_pool_bytes", _u64), ("slot_stride", _u64), ("windows", ctypes.POINTER(_vp)),
                ("n_windows", _u32), ("n_objects", _u32), ("window_bytes", _u64),
                ("objects", ctypes.POINTER(msi_object_desc)), ("source", ctypes.POINTER(msi_source_desc)),
                ("prefetch_slots", _u32), ("reserved1", _u32)]


class msi_ticket(ctypes.Structure):
    _fields_ = [("layer", _u32), ("expert", _u32), ("slot", _i32), ("generation", _u32),
                ("epoch", _u32), ("hit", _u32)]


class msi_routing(ctypes.Structure):
    _fields_ = [("idx", _vp), ("weights", _vp), ("counts", _vp), ("offsets", _vp), ("demand", _vp),
                ("perm", _vp), ("inv", _vp), ("row_weight", _vp)]


class msi_route_args(ctypes.Structure):
    _fields_ = [("n_tokens", _u32), ("reserved", _u32), ("x", _vp), ("w_router", _vp), ("bias", _vp),
                ("r", msi_routing), ("workspace", _vp), ("workspace_bytes", _u64)]


class msi_forward_args(ctypes.Structure):
    _fields_ = [("layer", _u32), ("n_tokens", _u32), ("x", _vp), ("r", msi_routing),
                ("shared_object", _vp), ("out", _vp), ("workspace", _vp), ("workspace_bytes", _u64)]


class msi_slot_info(ctypes.Structure):
    _fields_ = [("state", _u32), ("expert", _i32), ("generation", _u32), ("epoch", _u32),
                ("consumers", _u32), ("holds", _u32), ("last_use", _u64)]


class msi_stats(ctypes.Structure):
    _fields_ = [(n, _u64) for n in ("forwards", "rounds", "fills", "fills_published", "fills_discarded",
                                    "hits", "misses", "evictions", "h2d_bytes", "rejections",
                                    "stale_detected", "fills_in_flight", "windows_busy",
                                    "consumers_live")] + [("epoch", _u32), ("reserved", _u32),
                                                          ("prefetch_fills", _u64), ("prefetch_used", _u64)]


KERNEL_KINDS = ["router_logits", "topk", "permute", "gateup_tile", "gateup_stream", "down_tile",
                "down_stream", "expert_f32", "shared", "combine", "fill"]


class msi_timings(ctypes.Structure):
    _fields_ = [("launches", _u64 * len(KERNEL_KINDS)), ("ms", ctypes.c_double * len(KERNEL_KINDS))]


EXPORTS = ["msi_residual_init", "msi_residual_add", "msi_plan_set_timing", "msi_plan_set_timing_period",
           "msi_plan_timings", "msi_last_error", "msi_abi_version", "msi_plan_create", "msi_plan_destroy",
           "msi_plan_reset",
           "msi_workspace_size", "msi_slot_fill", "msi_plan_poll", "msi_route", "msi_moe_forward",
           "msi_moe_forward_noalloc",
           "msi_slot_hold", "msi_slot_unhold", "msi_slot_query", "msi_plan_stats",
           "msi_debug_set_device_gen", "msi_stream_threshold", "msi_source_stats_get",
           "msi_debug_source_fault", "msi_debug_source_release", "msi_prefetch"]


class MsiError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    L.msi_last_error.restype = ctypes.c_char_p
    L.msi_abi_version.restype = _u32
    L.msi_plan_create.argtypes = [P(msi_plan_desc), P(_vp)]
    L.msi_plan_destroy.argtypes = [_vp]
    L.msi_plan_reset.argtypes = [_vp]
    L.msi_workspace_size.argtypes = [_vp, _u32, P(_u64)]
    L.msi_slot_fill.argtypes = [_vp, _u32, _u32, _i32, _vp, P(msi_ticket)]
    L.msi_plan_poll.argtypes = [_vp]
    L.msi_route.argtypes = [_vp, P(msi_route_args), _vp]
    L.msi_moe_forward.argtypes = [_vp, P(msi_forward_args), _vp, _vp]
    L.msi_moe_forward_noalloc.argtypes = [_vp, P(msi_forward_args), _vp, _vp]
    L.msi_slot_hold.argtypes = [_vp, _u32, _u32]
    L.msi_slot_unhold.argtypes = [_vp, _u32, _u32]
    L.msi_slot_query.argtypes = [_vp, _u32, _u32, P(msi_slot_info)]
    L.msi_plan_stats.argtypes = [_vp, P(msi_stats)]
    L.msi_debug_set_device_gen.argtypes = [_vp, _u32, _u32, _u32]
    L.msi_source_stats_get.argtypes = [_vp, P(msi_source_stats)]
    L.msi_debug_source_fault.argtypes = [_vp, _u32, _u32, _u32, _u32]
    L.msi_debug_source_release.argtypes = [_vp]
    L.msi_prefetch.argtypes = [_vp, _u32, P(_i32), _u32, _vp, P(_u32)]
    L.msi_plan_set_timing.argtypes = [_vp, ctypes.c_int]
    L.msi_plan_set_timing_period.argtypes = [_vp, _u32]
    L.msi_residual_init.argtypes = [_vp, _vp, _vp, _u32, _u32, _vp]
    L.msi_residual_add.argtypes = [_vp, _vp, _vp, _u32, _u32, _vp]
    L.msi_plan_timings.argtypes = [_vp, P(msi_timings), ctypes.c_int]
    L.msi_stream_threshold.argtypes = [_u32]
    L.msi_stream_threshold.restype = _u32
    for n in EXPORTS:
        if n not in ("msi_last_error", "msi_abi_version", "msi_stream_threshold"):
            getattr(L, n).restype = _i32
    if L.msi_abi_version() != MSI_ABI_VERSION:
        raise ImportError("libmsi.so ABI version mismatch")
    return L


lib = _load()


def _check(status: int):
    if status != MSI_OK:
        raise MsiError(status, lib.msi_last_error().decode())


def last_error() -> str:
    return lib.msi_last_error().decode()


def stream_threshold(v: int = 0) -> int:
    return int(lib.msi_stream_threshold(v))


def residual_init(x0_bf16, h, x_bf16, stream=None):
    """h = float(x0); x = bf16(rmsnorm(h)) per row (bf16 bits in int16 tensors, h float32 [rows, cols])."""
    _check(lib.msi_residual_init(_ptr(x0_bf16), _ptr(h), _ptr(x_bf16), h.shape[0], h.shape[1], _stream(stream)))


def residual_add(out, h, x_bf16, stream=None):
    """h += out; x = bf16(rmsnorm(h)) per row."""
    _check(lib.msi_residual_add(_ptr(out), _ptr(h), _ptr(x_bf16), h.shape[0], h.shape[1], _stream(stream)))


# ---------------------------------------------------------------------------
# torch plumbing (allocation and streams only)
# ---------------------------------------------------------------------------

def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    return s.cuda_stream if hasattr(s, "cuda_stream") else int(s)


def object_nbytes(d: int, I: int, wdtype: str) -> int:
    if wdtype == "f32":
        return 3 * I * d * 4
    if wdtype == "bf16":
        return 3 * I * d * 2
    if wdtype == "kq":        # Wg, Wu in the 4.5-bit format, Wd in the 6.5625-bit format
        k4 = lambda r, c: r * c // 2 + r * (c // 256) * 16  # noqa: E731
        k6 = lambda r, c: r * c // 2 + r * c // 4 + r * c // 16 + r * (c // 256) * 2  # noqa: E731
        return 2 * k4(I, d) + k6(d, I)
    m = lambda r, c: r * c // 2 + r * (c // 32) * 2  # noqa: E731
    return 2 * m(I, d) + m(d, I)


@dataclass
class Routing:
    """Device arrays of one routing of T tokens (see msi_routing)."""
    idx: object
    weights: object
    counts: object
    offsets: object
    demand: object
    perm: object
    inv: object
    row_weight: object

    @staticmethod
    def alloc(T: int, K: int, E: int, device="cuda") -> "Routing":
        import torch
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        return Routing(idx=torch.empty((T, K), **i32), weights=torch.empty((T, K), **f32),
                       counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32),
                       demand=torch.empty(E + 1, **i32), perm=torch.empty(T * K, **i32), inv=torch.empty((T, K), **i32),
                       row_weight=torch.empty(T * K, **f32))

    def __setattr__(self, name, value):
        object.__setattr__(self, name, value)
        if name != "_c":
            object.__setattr__(self, "_c", None)     # arrays changed: marshal again

    def c(self) -> msi_routing:
        if getattr(self, "_c", None) is None:
            object.__setattr__(self, "_c", msi_routing(
                _ptr(self.idx), _ptr(self.weights), _ptr(self.counts), _ptr(self.offsets),
                _ptr(self.demand), _ptr(self.perm), _ptr(self.inv), _ptr(self.row_weight)))
        return self._c


class Plan:
    """One msi_plan plus the torch buffers it refers to (slot pool, windows).

    objects: sequence of (layer, expert, window, offset, nbytes).
    windows: pinned uint8 CPU tensors, all of the same size.
    source: None, or a Source (objects read from canonical files; windows
    are then its staging windows and ``objects`` must be empty).
    """

    def __init__(self, *, n_layers: int, n_experts: int, d_model: int, d_ff: int, top_k: int,
                 wdtype: str, slots_per_layer: int, windows: Sequence, objects: Sequence[Tuple],
                 transient_slots: int = 0, slot_stride: Optional[int] = None, device="cuda",
                 slot_pool=None, source: Optional["Source"] = None, policy: str = "lru",
                 prefetch_slots: int = 0):
        import torch
        self.wdtype = wdtype
        self.n_layers, self.n_experts, self.d, self.I, self.K = n_layers, n_experts, d_model, d_ff, top_k
        ob = object_nbytes(d_model, d_ff, wdtype)
        self.object_bytes = ob
        self.slot_stride = slot_stride or ((ob + 255) // 256) * 256
        self.pool_slots = slots_per_layer if slots_per_layer > 0 else (transient_slots or 8)
        pool_bytes = n_layers * self.pool_slots * self.slot_stride
        if slot_pool is None:
            slot_pool = torch.empty(pool_bytes + 256, dtype=torch.uint8, device=device)
        self._pool_tensor = slot_pool
        base = slot_pool.data_ptr()
        self.slot_pool_ptr = (base + 255) // 256 * 256
        self.slot_pool_bytes = slot_pool.numel() - (self.slot_pool_ptr - base)
        self.windows = list(windows)
        self.source = source
        if source is not None:
            self.windows = source.windows
        self._win_ptrs = (_vp * len(self.windows))(*[_window_ptr(w) for w in self.windows])
        self._objs = (msi_object_desc * max(1, len(objects)))(
            *[msi_object_desc(int(l), int(e), int(w), 0, int(o), int(n)) for (l, e, w, o, n) in objects])
        desc = msi_plan_desc(
            abi_version=MSI_ABI_VERSION, n_layers=n_layers, n_experts=n_experts, d_model=d_model,
            d_ff=d_ff, top_k=top_k, wdtype=WDTYPE[wdtype], slots_per_layer=slots_per_layer,
            transient_slots=transient_slots, policy=POLICIES[policy], slot_pool=self.slot_pool_ptr,
            slot_pool_bytes=self.slot_pool_bytes, slot_stride=self.slot_stride,
            windows=ctypes.cast(self._win_ptrs, ctypes.POINTER(_vp)), n_windows=len(self.windows),
            n_objects=len(objects),
            window_bytes=(source.window_bytes if source is not None else
                          (self.windows[0].numel() if self.windows else 0)),
            objects=ctypes.cast(self._objs, ctypes.POINTER(msi_object_desc)),
            source=ctypes.pointer(source.c()) if source is not None else None,
            prefetch_slots=prefetch_slots, reserved1=0)
        h = _vp()
        _check(lib.msi_plan_create(ctypes.byref(desc), ctypes.byref(h)))
        self.h = h

    # -- lifecycle --------------------------------------------------------------
    def close(self):
        if self.h:
            _check(lib.msi_plan_destroy(self.h))
            self.h = None

    def destroy_status(self) -> int:
        """msi_plan_destroy returning the status instead of raising."""
        st = lib.msi_plan_destroy(self.h)
        if st == MSI_OK:
            self.h = None
        return st

    def __del__(self):
        try:
            if getattr(self, "h", None):
                lib.msi_plan_destroy(self.h)
        except Exception:
            pass

    def reset(self):
        _check(lib.msi_plan_reset(self.h))

    def poll(self):
        _check(lib.msi_plan_poll(self.h))

    def workspace_size(self, T: int) -> int:
        n = _u64()
        _check(lib.msi_workspace_size(self.h, T, ctypes.byref(n)))
        return n.value

    def workspace(self, T: int, device="cuda"):
        import torch
        return torch.empty(self.workspace_size(T), dtype=torch.uint8, device=device)

    # -- C calls ----------------------------------------------------------------
    def slot_fill(self, layer: int, expert: int, slot: int = -1, side_stream=None) -> msi_ticket:
        t = msi_ticket()
        _check(lib.msi_slot_fill(self.h, layer, expert, slot, _stream(side_stream), ctypes.byref(t)))
        return t

    def route(self, x, w_router, bias, routing: Routing, workspace, stream=None):
        a = msi_route_args(n_tokens=x.shape[0], reserved=0, x=_ptr(x), w_router=_ptr(w_router),
                           bias=_ptr(bias), r=routing.c(), workspace=_ptr(workspace),
                           workspace_bytes=workspace.numel())
        _check(lib.msi_route(self.h, ctypes.byref(a), _stream(stream)))

    def forward_status(self, layer: int, x, routing: Routing, shared, out, workspace,
                       compute_stream=None, side_stream=None) -> int:
        a = msi_forward_args(layer=layer, n_tokens=x.shape[0], x=_ptr(x), r=routing.c(),
                             shared_object=_ptr(shared), out=_ptr(out), workspace=_ptr(workspace),
                             workspace_bytes=workspace.numel())
        return int(lib.msi_moe_forward(self.h, ctypes.byref(a), _stream(compute_stream), _stream(side_stream)))

    def forward_noalloc_status(self, layer: int, x, routing: Routing, shared, out, compute_stream=None,
                               side_stream=None) -> int:
        """msi_moe_forward_noalloc: the library's static scratch instead of a workspace."""
        a = msi_forward_args(layer=layer, n_tokens=x.shape[0], x=_ptr(x), r=routing.c(),
                             shared_object=_ptr(shared), out=_ptr(out), workspace=None, workspace_bytes=0)
        return int(lib.msi_moe_forward_noalloc(self.h, ctypes.byref(a), _stream(compute_stream),
                                               _stream(side_stream)))

    def forward(self, layer: int, x, routing: Routing, shared, out, workspace, compute_stream=None,
                side_stream=None):
        _check(self.forward_status(layer, x, routing, shared, out, workspace, compute_stream, side_stream))

    def prepare_step(self, layer: int, x, w_router, bias, routing: Routing, shared, out, workspace,
                     compute_stream=None, side_stream=None):
        """msi_route then msi_moe_forward on fixed buffers, with the argument
        structs built once: calling the result (no arguments) issues both
        calls and returns the forward's status.  For loops that reuse the same
        buffers, where rebuilding the structs on every call would be most of
        the host time between steps."""
        ra = msi_route_args(n_tokens=x.shape[0], reserved=0, x=_ptr(x), w_router=_ptr(w_router),
                            bias=_ptr(bias), r=routing.c(), workspace=_ptr(workspace),
                            workspace_bytes=workspace.numel())
        fa = msi_forward_args(layer=layer, n_tokens=x.shape[0], x=_ptr(x), r=routing.c(),
                              shared_object=_ptr(shared), out=_ptr(out), workspace=_ptr(workspace),
                              workspace_bytes=workspace.numel())
        h, cs, ss = self.h, _stream(compute_stream), _stream(side_stream)
        rp, fp = ctypes.byref(ra), ctypes.byref(fa)
        route, forward = lib.msi_route, lib.msi_moe_forward
        keep = (x, w_router, bias, routing, shared, out, workspace, ra, fa)   # buffers outlive the calls

        def step() -> int:
            _ = keep
            st = route(h, rp, cs)
            return st if st != MSI_OK else forward(h, fp, cs, ss)
        return step

    def hold(self, layer: int, slot: int):
        _check(lib.msi_slot_hold(self.h, layer, slot))

    def unhold(self, layer: int, slot: int):
        _check(lib.msi_slot_unhold(self.h, layer, slot))

    def query(self, layer: int, slot: int) -> msi_slot_info:
        i = msi_slot_info()
        _check(lib.msi_slot_query(self.h, layer, slot, ctypes.byref(i)))
        return i

    def stats(self) -> dict:
        s = msi_stats()
        _check(lib.msi_plan_stats(self.h, ctypes.byref(s)))
        return {n: getattr(s, n) for n, _ in msi_stats._fields_ if n != "reserved"}

    def set_timing_period(self, period: int):
        """Time only every period-th launch of each timed kind."""
        _check(lib.msi_plan_set_timing_period(self.h, period))

    def set_timing(self, enable=True, kinds=None):
        """Telemetry on/off; ``kinds`` (names of KERNEL_KINDS) restricts it."""
        v = int(bool(enable))
        if enable and kinds:
            v = 0
            for k in kinds:
                v |= 1 << KERNEL_KINDS.index(k)
            if v == 1:                      # kind 0 alone would read as "all"
                v |= 1 << 31
        _check(lib.msi_plan_set_timing(self.h, v))

    def timings(self, reset: bool = False) -> dict:
        """{kind: (launches, total_ms)} of the timing telemetry."""
        t = msi_timings()
        _check(lib.msi_plan_timings(self.h, ctypes.byref(t), int(bool(reset))))
        return {k: (int(t.launches[i]), float(t.ms[i])) for i, k in enumerate(KERNEL_KINDS)}

    def debug_set_device_gen(self, layer: int, slot: int, gen: int):
        _check(lib.msi_debug_set_device_gen(self.h, layer, slot, gen))

    def prefetch(self, layer: int, experts, side_stream=None) -> int:
        """msi_prefetch: fill the listed experts into the layer's prefetch bank; returns the fills issued."""
        ids = [int(e) for e in experts]
        arr = (_i32 * max(1, len(ids)))(*ids)
        n = _u32()
        _check(lib.msi_prefetch(self.h, layer, arr, len(ids), _stream(side_stream), ctypes.byref(n)))
        return n.value

    def source_stats(self) -> dict:
        s = msi_source_stats()
        _check(lib.msi_source_stats_get(self.h, ctypes.byref(s)))
        return {n: getattr(s, n) for n, _ in msi_source_stats._fields_}

    def source_fault(self, layer: int, expert: int, component: int, mode: str):
        """Test hook: the next read of that object's component is short / fails with EIO / is held."""
        _check(lib.msi_debug_source_fault(self.h, layer, expert, component, FAULTS[mode]))

    def source_release(self):
        _check(lib.msi_debug_source_release(self.h))


def _window_ptr(w) -> int:
    return w[1] if isinstance(w, tuple) else w.data_ptr()


class Source:
    """Canonical files plus the staging windows of a plan's source service.

    extents: (layer, expert, component, file, offset, nbytes) tuples;
    n_windows pinned staging windows of window_bytes (a multiple of align),
    each aligned to ``align``; inflight: reads in flight at most (1..8)."""

    def __init__(self, files: Sequence[str], extents: Sequence[Tuple], n_windows: int, window_bytes: int,
                 inflight: int, align: int = 4096, buffered_ok: bool = True):
        import torch
        self.files = [os.fsencode(f) for f in files]
        self.extents = list(extents)
        self.window_bytes = int(window_bytes)
        self.align = int(align)
        self.inflight = int(inflight)
        self.flags = MSI_SOURCE_BUFFERED_OK if buffered_ok else 0
        self._bufs, self.windows = [], []
        for _ in range(n_windows):
            b = torch.empty(self.window_bytes + self.align, dtype=torch.uint8, pin_memory=True)
            ptr = (b.data_ptr() + self.align - 1) // self.align * self.align
            self._bufs.append(b)
            self.windows.append((b, ptr))
        self._c = None

    def c(self) -> msi_source_desc:
        if self._c is None:
            self._fnames = (ctypes.c_char_p * len(self.files))(*self.files)
            self._ext = (msi_extent_desc * max(1, len(self.extents)))(
                *[msi_extent_desc(int(l), int(e), int(c), int(f), int(o), int(n))
                  for (l, e, c, f, o, n) in self.extents])
            self._c = msi_source_desc(files=self._fnames, n_files=len(self.files), inflight=self.inflight,
                                      flags=self.flags, align=self.align,
                                      extents=ctypes.cast(self._ext, ctypes.POINTER(msi_extent_desc)),
                                      n_extents=len(self.extents), reserved=0)
        return self._c


def pack_windows(objects: Sequence, per_window: int, layer: int = 0, first_expert: int = 0,
                 expert_ids: Optional[Sequence[int]] = None):
    """Copy expert objects (uint8 numpy arrays) into pinned host windows of
    ``per_window`` objects each.  Returns (windows, manifest entries)."""
    import numpy as np
    import torch
    objs = list(objects)
    ids = list(expert_ids) if expert_ids is not None else list(range(first_expert, first_expert + len(objs)))
    nb = objs[0].nbytes
    nwin = (len(objs) + per_window - 1) // per_window
    windows: List = []
    entries = []
    for w in range(nwin):
        buf = torch.empty(per_window * nb, dtype=torch.uint8, pin_memory=True)
        bnp = buf.numpy()
        for j in range(per_window):
            i = w * per_window + j
            if i >= len(objs):
                break
            bnp[j * nb:(j + 1) * nb] = np.asarray(objs[i], dtype=np.uint8)
            entries.append((layer, ids[i], w, j * nb, nb))
        windows.append(buf)
    return windows, entries
