"""TEST INFRASTRUCTURE ONLY: ctypes front end of the fp64 CPU oracle.

The oracle (``kvx_oracle.c``) computes the cross-model KV-translation
operator of the paper's Section 4 (the translation operator
KV^_B(C) = T_{A->B}(KV_A(C))) with the parameterised translator of Section 5,
as a plain fp64 loop nest; see ``kvx_oracle.h`` for the step list.

It shares no code with the GPU library and never imports it.  Inputs are any
object with the attributes of a problem instance (spec, src_k, src_v, w_k,
w_v, b_k, b_v, tgt_tokens, row_ptr, col_idx, weight, layer_map), or keyword
arrays; arrays are passed by pointer, read in their storage dtype and widened
exactly to double.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kvx_oracle.c")
LIB = os.path.join(HERE, "libkvx_oracle.so")

_lock = threading.Lock()
_lib = None


def build(out: str = LIB, src: str = SRC, extra=()) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC", *extra, src,
           "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


class _Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("rope_base", C.c_double), ("inv_freq", C.c_void_p)]


class _Problem(C.Structure):
    _fields_ = [("src", _Model), ("tgt", _Model), ("mix", C.c_int32),
                ("layer_map", C.c_void_p), ("dtype", C.c_int32),
                ("w_k", C.c_void_p), ("w_v", C.c_void_p),
                ("b_k", C.c_void_p), ("b_v", C.c_void_p),
                ("batch", C.c_int32), ("src_tokens", C.c_int32),
                ("src_k", C.c_void_p), ("src_v", C.c_void_p),
                ("tgt_tokens", C.c_void_p), ("row_ptr", C.c_void_p),
                ("col_idx", C.c_void_p), ("weight", C.c_void_p)]


def load(path: str = LIB):
    """Load (building first if absent) the oracle library."""
    global _lib
    with _lock:
        if path == LIB and _lib is not None:
            return _lib
        if not os.path.exists(path):
            build(path)
        lib = C.CDLL(path)
        lib.kvxo_rope.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_double,
                                  C.c_double, C.c_void_p]
        lib.kvxo_rope.restype = None
        lib.kvxo_rows.argtypes = [C.POINTER(_Problem), C.c_int64, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_void_p]
        lib.kvxo_rows.restype = C.c_int
        lib.kvxo_translate.argtypes = [C.POINTER(_Problem), C.c_int32, C.c_void_p,
                                       C.c_void_p]
        lib.kvxo_translate.restype = C.c_int
        lib.kvxo_num_threads.restype = C.c_int
        if path == LIB:
            _lib = lib
        return lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _model(shape, inv_freq, keep):
    inv = None
    if inv_freq is not None:
        inv = np.ascontiguousarray(inv_freq, dtype=np.float64)
        keep.append(inv)
    return _Model(shape.n_layers, shape.n_kv_heads, shape.head_dim,
                  float(shape.rope_base), _ptr(inv))


class _Bound:
    """A problem marshalled into the C struct (keeps its arrays alive)."""

    def __init__(self, prob, src_inv_freq=None, tgt_inv_freq=None):
        spec = prob.spec
        keep = []

        def arr(x, dt):
            if x is None:
                return None
            a = np.ascontiguousarray(x, dtype=dt)
            keep.append(a)
            return a

        sdt = np.float32 if spec.dtype == "f32" else np.uint16
        self.src_k = arr(prob.src_k, sdt)
        self.src_v = arr(prob.src_v, sdt)
        self.w_k = arr(prob.w_k, sdt)
        self.w_v = arr(prob.w_v, sdt)
        self.b_k = arr(prob.b_k, np.float32)
        self.b_v = arr(prob.b_v, np.float32)
        self.layer_map = arr(np.asarray(spec.layer_map), np.int32)
        ident = prob.row_ptr is None
        self.tgt_tokens = None if ident else arr(prob.tgt_tokens, np.int32)
        self.row_ptr = None if ident else arr(prob.row_ptr, np.int32)
        self.col_idx = None if ident else arr(prob.col_idx, np.int32)
        self.weight = None if ident else arr(prob.weight, np.float32)
        self.keep = keep
        self.spec = spec
        self.c = _Problem(
            _model(spec.src, src_inv_freq, keep), _model(spec.tgt, tgt_inv_freq, keep),
            spec.mix, _ptr(self.layer_map), 0 if spec.dtype == "f32" else 1,
            _ptr(self.w_k), _ptr(self.w_v), _ptr(self.b_k), _ptr(self.b_v),
            spec.batch, spec.src_tokens, _ptr(self.src_k), _ptr(self.src_v),
            _ptr(self.tgt_tokens), _ptr(self.row_ptr), _ptr(self.col_idx),
            _ptr(self.weight))


def rope(x, pos: float, base: float, inv_freq=None, lib_path: str = LIB) -> np.ndarray:
    """R(pos) x for one head vector (rotate-half pairing), fp64."""
    lib = load(lib_path)
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    inv = None if inv_freq is None else np.ascontiguousarray(inv_freq, dtype=np.float64)
    lib.kvxo_rope(x.ctypes.data, y.ctypes.data, x.shape[-1], float(pos), float(base),
                  _ptr(inv))
    return y


def translate(prob, cap=None, src_inv_freq=None, tgt_inv_freq=None, lib_path: str = LIB,
              out=None):
    """Full operator: returns (tgt_k, tgt_v), fp64 [Lt, B, Ht, cap, Dt].

    Rows t >= T_t[b] keep the initial contents of ``out`` (NaN by default)."""
    lib = load(lib_path)
    spec = prob.spec
    tt = np.asarray(prob.tgt_tokens)
    if cap is None:
        cap = int(tt.max()) if len(tt) else 0
    shape = (spec.tgt.n_layers, spec.batch, spec.tgt.n_kv_heads, cap, spec.tgt.head_dim)
    if out is None:
        tk = np.full(shape, np.nan)
        tv = np.full(shape, np.nan)
    else:
        tk, tv = out
    bp = _Bound(prob, src_inv_freq, tgt_inv_freq)
    rc = lib.kvxo_translate(C.byref(bp.c), int(cap), tk.ctypes.data, tv.ctypes.data)
    if rc:
        raise ValueError(f"oracle rejected the problem (code {rc})")
    return tk, tv


def rows(prob, layer, b, t, src_inv_freq=None, tgt_inv_freq=None, lib_path: str = LIB):
    """Selected output rows: returns (k, v), fp64 [n, Ht*Dt] (heads concatenated)."""
    lib = load(lib_path)
    spec = prob.spec
    layer = np.ascontiguousarray(layer, dtype=np.int32)
    b = np.ascontiguousarray(b, dtype=np.int32)
    t = np.ascontiguousarray(t, dtype=np.int32)
    n = len(layer)
    assert len(b) == n and len(t) == n
    dout = spec.tgt.n_kv_heads * spec.tgt.head_dim
    ok = np.empty((n, dout))
    ov = np.empty((n, dout))
    bp = _Bound(prob, src_inv_freq, tgt_inv_freq)
    rc = lib.kvxo_rows(C.byref(bp.c), n, layer.ctypes.data, b.ctypes.data, t.ctypes.data,
                       ok.ctypes.data, ov.ctypes.data)
    if rc:
        raise ValueError(f"oracle rejected the problem (code {rc})")
    return ok, ov


def num_threads(lib_path: str = LIB) -> int:
    return int(load(lib_path).kvxo_num_threads())
