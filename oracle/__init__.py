"""fp64 CPU oracle of the routed-expert MoE layer (ctypes over moe_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The product library never imports,
links or runs anything here, and this package imports nothing from the
product package.

Every function follows the plain definition written at the top of
``moe_oracle.c`` (router logits, top-K with lower-id tie-break, restricted
softmax, gated-SiLU experts, shared expert plus ascending-id combine, stable
counting-sort permutation, and the residual stream of a layer stack).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
LIB_PATH = os.path.join(_HERE, "libmsi_oracle.so")

DTYPE_CODE = {"f32": 0, "bf16": 1, "q4b32": 2, "kq": 3, "k4": 3, "k6": 4}
MAX_K = 64

_lib = None


def build(out: str = LIB_PATH, mutant: int = 0, quiet: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, IEEE semantics, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           f"-DMSIO_MUTANT={int(mutant)}", "-o", out, _SRC, "-lm"]
    subprocess.run(cmd, check=True, capture_output=quiet)
    return out


def _bind(lib):
    i64, i32, dbl = ctypes.c_int64, ctypes.c_int, ctypes.c_double
    vp = ctypes.c_void_p
    lib.msio_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.msio_bf16_to_f64.restype = dbl
    lib.msio_fp16_to_f64.argtypes = [ctypes.c_uint16]
    lib.msio_fp16_to_f64.restype = dbl
    lib.msio_f64_to_bf16.argtypes = [dbl]
    lib.msio_f64_to_bf16.restype = ctypes.c_uint16
    lib.msio_matrix_nbytes.argtypes = [i32, i64, i64]
    lib.msio_matrix_nbytes.restype = ctypes.c_size_t
    lib.msio_dequant.argtypes = [i32, i64, i64, vp, vp]
    lib.msio_router_logits.argtypes = [i64, i64, i64, i32, vp, vp, vp, vp]
    lib.msio_select_topk.argtypes = [i64, i64, i64, vp, vp, vp]
    lib.msio_gate_weights.argtypes = [i64, i64, i64, vp, vp, vp]
    lib.msio_permute.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp]
    lib.msio_expert_ffn.argtypes = [i64, i64, i32, vp, vp, vp, vp]
    lib.msio_moe_layer.argtypes = [i64, i64, i64, i64, i64, i32, i32, vp, vp, vp, vp, vp,
                                   i64, vp, vp, vp, vp, vp, vp, vp]
    lib.msio_residual_step.argtypes = [i64, i64, vp, vp, vp, vp]
    lib.msio_max_threads.restype = i32
    lib.msio_mutant.restype = i32
    return lib


def load(path: Optional[str] = None):
    """Load (building if absent) the oracle library.  ``path`` loads another
    build, e.g. a mutant compiled by the tests."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """Thin numpy front end; ``lib`` defaults to the clean build."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load()

    # -- stored-format upcasts ------------------------------------------------
    def bf16_to_f64(self, b: int) -> float:
        return self.lib.msio_bf16_to_f64(int(b))

    def fp16_to_f64(self, h: int) -> float:
        return self.lib.msio_fp16_to_f64(int(h))

    def f64_to_bf16(self, v: float) -> int:
        return int(self.lib.msio_f64_to_bf16(float(v)))

    def f64_to_bf16_array(self, a: np.ndarray) -> np.ndarray:
        f = self.lib.msio_f64_to_bf16
        return np.array([f(float(v)) for v in np.ravel(a)], dtype=np.uint16).reshape(np.shape(a))

    def dequant(self, dtype: str, rows: int, cols: int, src: np.ndarray) -> np.ndarray:
        src = np.ascontiguousarray(src)
        out = np.empty((rows, cols), dtype=np.float64)
        self.lib.msio_dequant(DTYPE_CODE[dtype], rows, cols, _p(src), _p(out))
        return out

    def matrix_nbytes(self, dtype: str, rows: int, cols: int) -> int:
        return int(self.lib.msio_matrix_nbytes(DTYPE_CODE[dtype], rows, cols))

    def expert_matrices(self, obj: np.ndarray, d: int, I: int, dtype: str):
        """(Wg [I,d], Wu [I,d], Wd [d,I]) of an expert object, as fp64."""
        nb = self.matrix_nbytes(dtype, I, d)
        obj = np.ascontiguousarray(obj, dtype=np.uint8)
        dd = "k6" if dtype == "kq" else dtype
        return (self.dequant(dtype, I, d, obj[:nb]),
                self.dequant(dtype, I, d, obj[nb:2 * nb]),
                self.dequant(dd, d, I, obj[2 * nb:]))

    # -- method steps -----------------------------------------------------------
    def router_logits(self, x: np.ndarray, wr: np.ndarray, bias: Optional[np.ndarray],
                      xdtype: str) -> np.ndarray:
        x = np.ascontiguousarray(x)
        wr = np.ascontiguousarray(wr)
        T, d = x.shape
        E = wr.shape[0]
        L = np.empty((T, E), dtype=np.float64)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        self.lib.msio_router_logits(T, d, E, DTYPE_CODE[xdtype], _p(x), _p(wr), _p(b), _p(L))
        return L

    def select_topk(self, L: np.ndarray, K: int):
        L = np.ascontiguousarray(L, dtype=np.float64)
        T, E = L.shape
        idx = np.empty((T, K), dtype=np.int32)
        gap = np.empty(T, dtype=np.float64)
        self.lib.msio_select_topk(T, E, K, _p(L), _p(idx), _p(gap))
        return idx, gap

    def gate_weights(self, L: np.ndarray, idx: np.ndarray) -> np.ndarray:
        L = np.ascontiguousarray(L, dtype=np.float64)
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        T, E = L.shape
        K = idx.shape[1]
        w = np.empty((T, K), dtype=np.float64)
        self.lib.msio_gate_weights(T, E, K, _p(L), _p(idx), _p(w))
        return w

    def permute(self, idx: np.ndarray, E: int):
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        T, K = idx.shape
        counts = np.empty(E, dtype=np.int32)
        offsets = np.empty(E + 1, dtype=np.int32)
        perm = np.empty(T * K, dtype=np.int32)
        inv = np.empty((T, K), dtype=np.int32)
        self.lib.msio_permute(T, E, K, _p(idx), _p(counts), _p(offsets), _p(perm), _p(inv))
        return counts, offsets, perm, inv

    def expert_ffn(self, obj: np.ndarray, x: np.ndarray, d: int, I: int, dtype: str) -> np.ndarray:
        obj = np.ascontiguousarray(obj, dtype=np.uint8)
        x = np.ascontiguousarray(x, dtype=np.float64)
        y = np.empty(d, dtype=np.float64)
        self.lib.msio_expert_ffn(d, I, DTYPE_CODE[dtype], _p(obj), _p(x), _p(y), None)
        return y

    def moe_layer(self, x: np.ndarray, wr: np.ndarray, bias: Optional[np.ndarray],
                  experts: Sequence[np.ndarray], shared: Optional[np.ndarray],
                  K: int, I: int, wdtype: str, xdtype: str,
                  tokens: Optional[Sequence[int]] = None,
                  forced_idx: Optional[np.ndarray] = None,
                  want_logits: bool = False):
        """Steps 1-5 for ``tokens`` (default all).  Returns a dict with
        out [n, d], idx [n, K], w [n, K], gap [n] (NaN when forced) and
        optionally logits [n, E]."""
        x = np.ascontiguousarray(x)
        wr = np.ascontiguousarray(wr)
        T, d = x.shape
        E = wr.shape[0]
        assert K <= MAX_K and len(experts) == E
        tok = None if tokens is None else np.ascontiguousarray(tokens, dtype=np.int64)
        n = T if tok is None else len(tok)
        # entries may be None for experts the caller knows are not selected;
        # a selected missing object turns that token's output into NaN
        objs = [None if o is None else np.ascontiguousarray(o, dtype=np.uint8) for o in experts]
        ptrs = (ctypes.c_void_p * E)(*[0 if o is None else o.ctypes.data for o in objs])
        sh = None if shared is None else np.ascontiguousarray(shared, dtype=np.uint8)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        fi = None if forced_idx is None else np.ascontiguousarray(forced_idx, dtype=np.int32)
        out = np.empty((n, d), dtype=np.float64)
        idx = np.empty((n, K), dtype=np.int32)
        w = np.empty((n, K), dtype=np.float64)
        gap = np.empty(n, dtype=np.float64)
        lg = np.empty((n, E), dtype=np.float64) if want_logits else None
        self.lib.msio_moe_layer(T, d, E, K, I, DTYPE_CODE[wdtype], DTYPE_CODE[xdtype],
                                _p(x), _p(wr), _p(b), ctypes.cast(ptrs, ctypes.c_void_p),
                                _p(sh), n, _p(tok), _p(fi), _p(out), _p(idx), _p(w), _p(gap),
                                _p(lg))
        res = {"out": out, "idx": idx, "w": w, "gap": gap}
        if want_logits:
            res["logits"] = lg
        return res

    def residual_step(self, h: np.ndarray, out: Optional[np.ndarray] = None):
        """Step 6 for one layer boundary: h_next = h + out (out None: h_next =
        h), x_next = bf16 bits of h_next / rms(h_next) per row.  Returns
        (h_next fp64, x_next uint16)."""
        h = np.ascontiguousarray(h, dtype=np.float64)
        rows, cols = h.shape
        o = None if out is None else np.ascontiguousarray(out, dtype=np.float64)
        hn = np.empty_like(h)
        x = np.empty((rows, cols), dtype=np.uint16)
        self.lib.msio_residual_step(rows, cols, _p(h), _p(o), _p(hn), _p(x))
        return hn, x

    def stack(self, h0: np.ndarray, layers: Sequence[dict], K: int, I: int, wdtype: str):
        """Step 6 over a stack: h_0 = h0 (fp64 [T, d]); layer l reads x_l =
        bf16(h_l / rms(h_l)) and h_{l+1} = h_l + out_l(x_l).  ``layers`` holds
        per layer dict(wr, bias, experts, shared).  Returns dict with h (the
        final residual stream), xs (each layer's bf16 input), idx and gap
        (each layer's selection and top-K logit gap)."""
        h, x = self.residual_step(h0)
        xs, idxs, gaps = [], [], []
        for ly in layers:
            r = self.moe_layer(x, ly["wr"], ly["bias"], ly["experts"], ly["shared"], K, I, wdtype, "bf16")
            xs.append(x)
            idxs.append(r["idx"])
            gaps.append(r["gap"])
            h, x = self.residual_step(h, r["out"])
        return {"h": h, "x": x, "xs": xs, "idx": idxs, "gap": gaps}

    def max_threads(self) -> int:
        return int(self.lib.msio_max_threads())
