"""Python binding of ``libkvx.so`` (argument marshalling only).

The entry points carry the C names -- ``kvx_plan_create``,
``kvx_plan_create_factored``, ``kvx_translate``, ``kvx_plan_destroy``
(include/kvx.h) and ``kvx_fit_create``,
``kvx_fit_accumulate``, ``kvx_fit_solve``, ``kvx_fit_reset``,
``kvx_fit_destroy`` (include/kvx_fit.h) -- and take torch tensors for device
buffers (torch provides device memory and streams; it computes nothing here).
Every step of the translation and of the fit runs in the library's HIP
kernels.

The library must have been built (``python -m paper_2608_30963_amd.build``);
loading fails loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvx.so")

KVX_OK, KVX_EINVAL, KVX_ESHAPE, KVX_EUNSUPPORTED, KVX_ENOMEM, KVX_EHIP, KVX_EDATA = range(7)
KVX_F32, KVX_BF16 = 0, 1
KVX_PREC_BF16X2, KVX_PREC_BF16, KVX_PREC_F16, KVX_PREC_BF16X2_OUTLIER = 0, 1, 2, 3
KVX_FACTORS_LOWRANK, KVX_FACTORS_MIXTURE = 1, 2
KVX_STAGE_POOL, KVX_STAGE_PROJECT, KVX_STAGE_STORE, KVX_STAGE_ALL = 1, 2, 4, 7

# Exported C symbols, as declared in include/kvx.h and include/kvx_fit.h.
SYMBOLS = ("kvx_plan_create", "kvx_plan_create_factored", "kvx_translate", "kvx_plan_destroy",
           "kvx_status_string",
           "kvx_last_hip_error", "kvx_plan_query", "kvx_staged_workspace_bytes",
           "kvx_translate_staged", "kvx_fit_create", "kvx_fit_accumulate",
           "kvx_fit_solve", "kvx_fit_solve_noalloc", "kvx_fit_reset", "kvx_fit_rows",
           "kvx_fit_query", "kvx_fit_destroy")


class KvxError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


class Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("rope_base", C.c_double), ("inv_freq", C.c_void_p)]


class PlanDesc(C.Structure):
    _fields_ = [("src", Model), ("tgt", Model), ("mix", C.c_int32),
                ("layer_map", C.c_void_p), ("dtype", C.c_int32),
                ("w_k", C.c_void_p), ("w_v", C.c_void_p),
                ("b_k", C.c_void_p), ("b_v", C.c_void_p), ("precision", C.c_int32),
                ("outlier_k", C.c_void_p), ("outlier_v", C.c_void_p)]


class Factors(C.Structure):
    _fields_ = [("kind", C.c_int32), ("rank", C.c_int32), ("u_k", C.c_void_p),
                ("u_v", C.c_void_p), ("v_k", C.c_void_p), ("v_v", C.c_void_p),
                ("n_mix", C.c_int32), ("alpha", C.c_void_p), ("w_k", C.c_void_p),
                ("w_v", C.c_void_p), ("b_k", C.c_void_p), ("b_v", C.c_void_p)]


class IO(C.Structure):
    _fields_ = [("batch", C.c_int32), ("src_tokens", C.c_int32),
                ("src_k", C.c_void_p), ("src_v", C.c_void_p), ("src_stride", C.c_int64 * 4),
                ("tgt_tokens", C.c_void_p), ("row_ptr", C.c_void_p),
                ("col_idx", C.c_void_p), ("weight", C.c_void_p),
                ("tgt_k", C.c_void_p), ("tgt_v", C.c_void_p), ("tgt_stride", C.c_int64 * 4),
                ("tgt_capacity", C.c_int32), ("block_table", C.c_void_p),
                ("block_size", C.c_int32), ("max_blocks", C.c_int32), ("num_blocks", C.c_int32)]


class FitDesc(C.Structure):
    _fields_ = [("src", Model), ("tgt", Model), ("mix", C.c_int32),
                ("layer_map", C.c_void_p), ("dtype", C.c_int32), ("fit_bias", C.c_int32)]


class FitIO(C.Structure):
    _fields_ = [("batch", C.c_int32), ("src_tokens", C.c_int32),
                ("src_k", C.c_void_p), ("src_v", C.c_void_p), ("src_stride", C.c_int64 * 4),
                ("tgt_tokens", C.c_void_p), ("row_ptr", C.c_void_p),
                ("col_idx", C.c_void_p), ("weight", C.c_void_p),
                ("tgt_k", C.c_void_p), ("tgt_v", C.c_void_p), ("tgt_stride", C.c_int64 * 4),
                ("tgt_capacity", C.c_int32)]


class FitInfo(C.Structure):
    _fields_ = [("systems", C.c_int32), ("n", C.c_int32), ("gram_blocks", C.c_int32),
                ("gram_launches", C.c_int32), ("rows", C.c_int64),
                ("device_bytes", C.c_int64), ("gram_ms", C.c_double)]


class PlanInfo(C.Structure):
    _fields_ = [("kernel", C.c_int32), ("tile_rows", C.c_int32), ("tile_cols", C.c_int32),
                ("threads", C.c_int32), ("precision", C.c_int32), ("weight_bytes", C.c_int64),
                ("split_ksteps", C.c_int64), ("ksteps", C.c_int64),
                ("tile_order", C.c_int32)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libkvx.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2608_30963_amd.build` (no fallback exists)")
    # torch provides the device memory and streams; its HIP runtime must be
    # the process's only one, so it is loaded before the library binds to
    # whichever runtime is already present
    import torch  # noqa: F401
    lib = C.CDLL(path)
    lib.kvx_plan_create.argtypes = [C.POINTER(PlanDesc), C.POINTER(C.c_void_p)]
    lib.kvx_plan_create.restype = C.c_int
    lib.kvx_plan_create_factored.argtypes = [C.POINTER(PlanDesc), C.POINTER(Factors),
                                             C.POINTER(C.c_void_p)]
    lib.kvx_plan_create_factored.restype = C.c_int
    lib.kvx_translate.argtypes = [C.c_void_p, C.POINTER(IO), C.c_void_p]
    lib.kvx_translate.restype = C.c_int
    lib.kvx_plan_destroy.argtypes = [C.c_void_p]
    lib.kvx_plan_destroy.restype = None
    lib.kvx_status_string.argtypes = [C.c_int]
    lib.kvx_status_string.restype = C.c_char_p
    lib.kvx_last_hip_error.restype = C.c_int32
    lib.kvx_plan_query.argtypes = [C.c_void_p, C.POINTER(PlanInfo)]
    lib.kvx_plan_query.restype = C.c_int
    lib.kvx_staged_workspace_bytes.argtypes = [C.c_void_p, C.POINTER(IO), C.c_int32,
                                               C.POINTER(C.c_size_t)]
    lib.kvx_staged_workspace_bytes.restype = C.c_int
    lib.kvx_translate_staged.argtypes = [C.c_void_p, C.POINTER(IO), C.c_void_p, C.c_size_t,
                                         C.c_uint32, C.c_void_p]
    lib.kvx_translate_staged.restype = C.c_int
    lib.kvx_fit_create.argtypes = [C.POINTER(FitDesc), C.POINTER(C.c_void_p)]
    lib.kvx_fit_create.restype = C.c_int
    lib.kvx_fit_accumulate.argtypes = [C.c_void_p, C.POINTER(FitIO), C.c_void_p]
    lib.kvx_fit_accumulate.restype = C.c_int
    lib.kvx_fit_solve.argtypes = [C.c_void_p, C.c_double, C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_void_p]
    lib.kvx_fit_solve.restype = C.c_int
    lib.kvx_fit_solve_noalloc.argtypes = lib.kvx_fit_solve.argtypes
    lib.kvx_fit_solve_noalloc.restype = C.c_int
    lib.kvx_fit_reset.argtypes = [C.c_void_p, C.c_void_p]
    lib.kvx_fit_reset.restype = C.c_int
    lib.kvx_fit_rows.argtypes = [C.c_void_p]
    lib.kvx_fit_rows.restype = C.c_int64
    lib.kvx_fit_query.argtypes = [C.c_void_p, C.POINTER(FitInfo)]
    lib.kvx_fit_query.restype = C.c_int
    lib.kvx_fit_destroy.argtypes = [C.c_void_p]
    lib.kvx_fit_destroy.restype = None
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().kvx_status_string(int(status)).decode()


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    return int(t)


def _host_array(values, ctype):
    if values is None:
        return None
    vals = list(values)
    return (ctype * max(1, len(vals)))(*vals)


@dataclass
class ModelShape:
    n_layers: int
    n_kv_heads: int
    head_dim: int
    rope_base: float


def _model(m, inv_freq, keep) -> Model:
    inv = None
    if inv_freq is not None:
        inv = _host_array([float(x) for x in inv_freq], C.c_double)
        keep.append(inv)
    return Model(int(m.n_layers), int(m.n_kv_heads), int(m.head_dim), float(m.rope_base),
                 C.cast(inv, C.c_void_p).value if inv is not None else None)


def _marks(arr, src, keep):
    """Host outlier marks [Ls][Hs][Ds] (any array-like, nonzero = marked) as a
    uint8 buffer, or None."""
    if arr is None:
        return None
    import numpy as np
    a = np.ascontiguousarray(np.asarray(arr) != 0, dtype=np.uint8)
    want = (int(src.n_layers), int(src.n_kv_heads), int(src.head_dim))
    if a.shape != want:
        raise ValueError(f"outlier marks have shape {a.shape}, expected {want}")
    buf = (C.c_uint8 * a.size).from_buffer_copy(a.tobytes())
    keep.append(buf)
    return C.cast(buf, C.c_void_p).value


def kvx_plan_create(src, tgt, mix: int, layer_map: Sequence[int], dtype: int, w_k, w_v,
                    b_k=None, b_v=None, precision: int = KVX_PREC_BF16X2,
                    src_inv_freq=None, tgt_inv_freq=None, outlier_k=None,
                    outlier_v=None) -> int:
    """Create a plan; returns the opaque handle (an int).  ``w_k``/``w_v``/
    ``b_k``/``b_v`` are device tensors (or raw device pointers);
    ``outlier_k``/``outlier_v`` host marks [Ls][Hs][Ds] for precision
    KVX_PREC_BF16X2_OUTLIER."""
    lib = load()
    keep = []
    lm = _host_array([int(x) for x in layer_map], C.c_int32)
    keep.append(lm)
    desc = PlanDesc(_model(src, src_inv_freq, keep), _model(tgt, tgt_inv_freq, keep),
                    int(mix), C.cast(lm, C.c_void_p).value, int(dtype), _ptr(w_k), _ptr(w_v),
                    _ptr(b_k), _ptr(b_v), int(precision), _marks(outlier_k, src, keep),
                    _marks(outlier_v, src, keep))
    h = C.c_void_p()
    st = lib.kvx_plan_create(C.byref(desc), C.byref(h))
    if st != KVX_OK:
        raise KvxError(st, "kvx_plan_create")
    return h.value


def kvx_plan_create_factored(src, tgt, mix: int, layer_map: Sequence[int], dtype: int,
                             lowrank=None, mixture=None, b_k=None, b_v=None,
                             precision: int = KVX_PREC_BF16X2, src_inv_freq=None,
                             tgt_inv_freq=None) -> int:
    """Create a plan from translator factors; returns the handle.
    ``lowrank=(u_k, v_k, u_v, v_v)`` (device [Lt][dout][r], [Lt][r][din];
    ``b_k``/``b_v`` give its bias) or ``mixture=(alpha, w_k, w_v, b_k, b_v)``
    (host alpha [K]; device [K][Lt][dout][din] and fp32 [K][Lt][dout] or
    None)."""
    lib = load()
    keep = []
    lm = _host_array([int(x) for x in layer_map], C.c_int32)
    keep.append(lm)
    f = Factors()
    if lowrank is not None:
        u_k, v_k, u_v, v_v = lowrank
        f.kind = KVX_FACTORS_LOWRANK
        f.rank = int(u_k.shape[-1]) if hasattr(u_k, "shape") else 0
        f.u_k, f.v_k, f.u_v, f.v_v = _ptr(u_k), _ptr(v_k), _ptr(u_v), _ptr(v_v)
    elif mixture is not None:
        alpha, w_k, w_v, mb_k, mb_v = mixture
        al = _host_array([float(x) for x in alpha], C.c_double)
        keep.append(al)
        f.kind = KVX_FACTORS_MIXTURE
        f.n_mix = len(alpha)
        f.alpha = C.cast(al, C.c_void_p).value
        f.w_k, f.w_v, f.b_k, f.b_v = _ptr(w_k), _ptr(w_v), _ptr(mb_k), _ptr(mb_v)
    desc = PlanDesc(_model(src, src_inv_freq, keep), _model(tgt, tgt_inv_freq, keep),
                    int(mix), C.cast(lm, C.c_void_p).value, int(dtype), None, None,
                    _ptr(b_k), _ptr(b_v), int(precision))
    h = C.c_void_p()
    st = lib.kvx_plan_create_factored(C.byref(desc), C.byref(f), C.byref(h))
    if st != KVX_OK:
        raise KvxError(st, "kvx_plan_create_factored")
    return h.value


def make_io(batch: int, src_tokens: int, src_k, src_v, tgt_k, tgt_v, tgt_capacity: int,
            tgt_tokens=None, row_ptr=None, col_idx=None, weight=None,
            src_stride=(0, 0, 0, 0), tgt_stride=(0, 0, 0, 0), block_table=None,
            block_size: int = 0, max_blocks: int = 0, num_blocks: int = 0):
    """Build the kvx_io struct; returns (io, keepalive).  ``block_table``
    (device int32 [batch][max_blocks]) selects the paged target layout."""
    keep = []
    tt = None
    if tgt_tokens is not None:
        tt = _host_array([int(x) for x in tgt_tokens], C.c_int32)
        keep.append(tt)
    io = IO(int(batch), int(src_tokens), _ptr(src_k), _ptr(src_v),
            (C.c_int64 * 4)(*[int(x) for x in src_stride]),
            C.cast(tt, C.c_void_p).value if tt is not None else None,
            _ptr(row_ptr), _ptr(col_idx), _ptr(weight), _ptr(tgt_k), _ptr(tgt_v),
            (C.c_int64 * 4)(*[int(x) for x in tgt_stride]), int(tgt_capacity),
            _ptr(block_table), int(block_size), int(max_blocks), int(num_blocks))
    return io, keep


def kvx_translate(plan: int, io: IO, stream=None) -> int:
    """Enqueue a translation; ``stream`` is a torch stream, a raw hipStream_t
    (int) or None (the current torch stream)."""
    lib = load()
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    st = lib.kvx_translate(C.c_void_p(plan), C.byref(io), C.c_void_p(handle))
    if st != KVX_OK:
        raise KvxError(st, "kvx_translate")
    return st


def kvx_translate_status(plan, io: IO, stream_handle: int = 0) -> int:
    """Raw status of kvx_translate (no exception)."""
    return int(load().kvx_translate(C.c_void_p(plan), C.byref(io), C.c_void_p(stream_handle)))


def kvx_staged_workspace_bytes(plan: int, io: IO, layers: int) -> int:
    """Device bytes the staged translation's workspace needs for `layers`
    target layers of this call."""
    n = C.c_size_t(0)
    st = load().kvx_staged_workspace_bytes(C.c_void_p(plan), C.byref(io), int(layers),
                                           C.byref(n))
    if st != KVX_OK:
        raise KvxError(st, "kvx_staged_workspace_bytes")
    return int(n.value)


def kvx_translate_staged_status(plan: int, io: IO, workspace: int, workspace_bytes: int,
                                stages: int = KVX_STAGE_ALL, stream_handle: int = 0) -> int:
    """Raw status of kvx_translate_staged (no exception); `workspace` is a
    device address."""
    return int(load().kvx_translate_staged(C.c_void_p(plan), C.byref(io), C.c_void_p(workspace),
                                           int(workspace_bytes), int(stages),
                                           C.c_void_p(stream_handle)))


def kvx_translate_staged(plan: int, io: IO, workspace, workspace_bytes: Optional[int] = None,
                         stages: int = KVX_STAGE_ALL, stream=None) -> int:
    """Enqueue the staged (three-launch) translation; `workspace` is a device
    tensor (its size is passed unless `workspace_bytes` is given) or a
    device address."""
    if hasattr(workspace, "data_ptr"):
        nbytes = workspace.numel() * workspace.element_size()
        ptr = workspace.data_ptr()
    else:
        nbytes, ptr = workspace_bytes, int(workspace)
    if workspace_bytes is not None:
        nbytes = workspace_bytes
    st = kvx_translate_staged_status(plan, io, ptr, nbytes, stages, _stream_handle(stream))
    if st != KVX_OK:
        raise KvxError(st, "kvx_translate_staged")
    return st


def kvx_plan_destroy(plan: Optional[int]) -> None:
    load().kvx_plan_destroy(C.c_void_p(plan) if plan else None)


def kvx_plan_query(plan: int) -> PlanInfo:
    info = PlanInfo()
    st = load().kvx_plan_query(C.c_void_p(plan), C.byref(info))
    if st != KVX_OK:
        raise KvxError(st, "kvx_plan_query")
    return info


class Translator:
    """RAII wrapper around a plan, for the tests and the benchmark."""

    def __init__(self, src, tgt, mix, layer_map, dtype, w_k=None, w_v=None, b_k=None,
                 b_v=None, precision=KVX_PREC_BF16X2, src_inv_freq=None, tgt_inv_freq=None,
                 lowrank=None, mixture=None, outlier_k=None, outlier_v=None):
        """Dense translator from ``w_k``/``w_v``, or a composed one from
        ``lowrank`` / ``mixture`` (see kvx_plan_create_factored)."""
        self.src, self.tgt, self.mix = src, tgt, mix
        self.dtype = dtype
        self.plan = None
        if lowrank is not None or mixture is not None:
            self.plan = kvx_plan_create_factored(src, tgt, mix, layer_map, dtype, lowrank,
                                                 mixture, b_k, b_v, precision, src_inv_freq,
                                                 tgt_inv_freq)
        else:
            self.plan = kvx_plan_create(src, tgt, mix, layer_map, dtype, w_k, w_v, b_k, b_v,
                                        precision, src_inv_freq, tgt_inv_freq, outlier_k,
                                        outlier_v)

    def info(self) -> PlanInfo:
        return kvx_plan_query(self.plan)

    def __call__(self, src_k, src_v, tgt_k, tgt_v, tgt_capacity=None, tgt_tokens=None,
                 row_ptr=None, col_idx=None, weight=None, stream=None,
                 src_stride=(0, 0, 0, 0), tgt_stride=(0, 0, 0, 0), block_table=None,
                 block_size=0):
        """Contiguous targets [Lt][B][Ht][cap][Dt]; with ``block_table``
        ([B][max_blocks] int32 on the device) paged targets
        [Lt][num_blocks][Ht][block_size][Dt] (or the given strides)."""
        batch, src_tokens = int(src_k.shape[1]), int(src_k.shape[3])
        max_blocks = num_blocks = 0
        if block_table is not None:
            max_blocks, num_blocks = int(block_table.shape[1]), int(tgt_k.shape[1])
            cap = 0 if tgt_capacity is None else int(tgt_capacity)
        else:
            cap = int(tgt_k.shape[3]) if tgt_capacity is None else int(tgt_capacity)
        io, keep = make_io(batch, src_tokens, src_k, src_v, tgt_k, tgt_v, cap, tgt_tokens,
                           row_ptr, col_idx, weight, src_stride, tgt_stride, block_table,
                           block_size, max_blocks, num_blocks)
        kvx_translate(self.plan, io, stream)
        del keep

    def close(self):
        if self.plan:
            kvx_plan_destroy(self.plan)
            self.plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# Translator fit (include/kvx_fit.h)
# ---------------------------------------------------------------------------

def _stream_handle(stream) -> int:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def kvx_fit_create(src, tgt, mix: int, layer_map: Sequence[int], dtype: int,
                   fit_bias: bool = True, src_inv_freq=None, tgt_inv_freq=None) -> int:
    lib = load()
    keep = []
    lm = _host_array([int(x) for x in layer_map], C.c_int32)
    keep.append(lm)
    desc = FitDesc(_model(src, src_inv_freq, keep), _model(tgt, tgt_inv_freq, keep), int(mix),
                   C.cast(lm, C.c_void_p).value, int(dtype), 1 if fit_bias else 0)
    h = C.c_void_p()
    st = lib.kvx_fit_create(C.byref(desc), C.byref(h))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_create")
    return h.value


def make_fit_io(batch: int, src_tokens: int, src_k, src_v, tgt_k, tgt_v, tgt_capacity: int,
                tgt_tokens=None, row_ptr=None, col_idx=None, weight=None,
                src_stride=(0, 0, 0, 0), tgt_stride=(0, 0, 0, 0)):
    keep = []
    tt = None
    if tgt_tokens is not None:
        tt = _host_array([int(x) for x in tgt_tokens], C.c_int32)
        keep.append(tt)
    io = FitIO(int(batch), int(src_tokens), _ptr(src_k), _ptr(src_v),
               (C.c_int64 * 4)(*[int(x) for x in src_stride]),
               C.cast(tt, C.c_void_p).value if tt is not None else None,
               _ptr(row_ptr), _ptr(col_idx), _ptr(weight), _ptr(tgt_k), _ptr(tgt_v),
               (C.c_int64 * 4)(*[int(x) for x in tgt_stride]), int(tgt_capacity))
    return io, keep


def kvx_fit_accumulate(fit: int, io: FitIO, stream=None) -> int:
    st = load().kvx_fit_accumulate(C.c_void_p(fit), C.byref(io), C.c_void_p(_stream_handle(stream)))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_accumulate")
    return st


def kvx_fit_solve(fit: int, lam: float, w_k, w_v, b_k=None, b_v=None, stream=None) -> int:
    st = load().kvx_fit_solve(C.c_void_p(fit), float(lam), _ptr(w_k), _ptr(w_v), _ptr(b_k),
                              _ptr(b_v), C.c_void_p(_stream_handle(stream)))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_solve")
    return st


def kvx_fit_solve_noalloc(fit: int, lam: float, w_k, w_v, b_k=None, b_v=None,
                          stream=None) -> int:
    st = load().kvx_fit_solve_noalloc(C.c_void_p(fit), float(lam), _ptr(w_k), _ptr(w_v),
                                      _ptr(b_k), _ptr(b_v), C.c_void_p(_stream_handle(stream)))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_solve_noalloc")
    return st


def kvx_fit_reset(fit: int, stream=None) -> int:
    st = load().kvx_fit_reset(C.c_void_p(fit), C.c_void_p(_stream_handle(stream)))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_reset")
    return st


def kvx_fit_rows(fit: int) -> int:
    return int(load().kvx_fit_rows(C.c_void_p(fit)))


def kvx_fit_query(fit: int) -> FitInfo:
    info = FitInfo()
    st = load().kvx_fit_query(C.c_void_p(fit), C.byref(info))
    if st != KVX_OK:
        raise KvxError(st, "kvx_fit_query")
    return info


def kvx_fit_destroy(fit: Optional[int]) -> None:
    load().kvx_fit_destroy(C.c_void_p(fit) if fit else None)


class Fitter:
    """RAII wrapper around a fit, for the tests and the benchmark."""

    def __init__(self, src, tgt, mix, layer_map, dtype, fit_bias=True, src_inv_freq=None,
                 tgt_inv_freq=None):
        self.tgt, self.mix, self.src = tgt, mix, src
        self.fit_bias = fit_bias
        self.handle = kvx_fit_create(src, tgt, mix, layer_map, dtype, fit_bias, src_inv_freq,
                                     tgt_inv_freq)

    def accumulate(self, src_k, src_v, tgt_k, tgt_v, tgt_tokens=None, row_ptr=None,
                   col_idx=None, weight=None, stream=None, src_stride=(0, 0, 0, 0),
                   tgt_stride=(0, 0, 0, 0)):
        """Source caches [Ls][B][Hs][T_s][Ds], native target caches
        [Lt][B][Ht][cap][Dt] (torch device tensors)."""
        batch, src_tokens = int(src_k.shape[1]), int(src_k.shape[3])
        io, keep = make_fit_io(batch, src_tokens, src_k, src_v, tgt_k, tgt_v,
                               int(tgt_k.shape[3]), tgt_tokens, row_ptr, col_idx, weight,
                               src_stride, tgt_stride)
        kvx_fit_accumulate(self.handle, io, stream)
        del keep

    def solve(self, lam, stream=None, noalloc=False):
        """Returns fp32 device tensors (w_k, w_v, b_k, b_v); ``noalloc``
        solves through kvx_fit_solve_noalloc."""
        import torch
        Lt = self.tgt.n_layers
        dout = self.tgt.n_kv_heads * self.tgt.head_dim
        din = self.mix * self.src.n_kv_heads * self.src.head_dim
        w_k = torch.empty((Lt, dout, din), dtype=torch.float32, device="cuda")
        w_v = torch.empty_like(w_k)
        b_k = torch.empty((Lt, dout), dtype=torch.float32, device="cuda")
        b_v = torch.empty_like(b_k)
        (kvx_fit_solve_noalloc if noalloc else kvx_fit_solve)(self.handle, lam, w_k, w_v, b_k,
                                                                b_v, stream)
        return w_k, w_v, b_k, b_v

    def reset(self, stream=None):
        kvx_fit_reset(self.handle, stream)

    @property
    def rows(self) -> int:
        return kvx_fit_rows(self.handle)

    def info(self) -> FitInfo:
        return kvx_fit_query(self.handle)

    def close(self):
        if self.handle:
            kvx_fit_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
