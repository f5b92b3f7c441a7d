"""Seeded synthetic inputs for the KV-translation operator.

This module only *draws* inputs; it holds none of the operator's arithmetic
(no RoPE, no pooling, no projection).  Both the GPU path and the CPU oracle
consume exactly the arrays produced here, so they see identical bits.

Shapes follow the model pairs of the paper's evaluation (Section 6.1, "Model
configurations": Qwen2.5-7B -> Qwen2.5-1.5B, Qwen2.5-1.5B -> Gemma-2-2B,
Llama3.1-70B -> Qwen2.5-7B) at the KV-cache level: layers, KV heads,
head_dim and RoPE base of each model.  The paper's datasets (NoLiMa,
LongBench2, FineWeb-Edu) and trained translators are not available; seeded
Gaussian KV caches and Gaussian translator weights stand in for them.

Random streams (numpy PCG64, seeded with a tuple so every slice can be drawn
independently):

    (seed, cfg, 0, layer, b)  source K slice [Hs, T, Ds]
    (seed, cfg, 1, layer, b)  source V slice
    (seed, cfg, 2, layer)     outlier channels of K, per head
    (seed, cfg, 3, layer)     outlier channels of V, per head
    (seed, cfg, 4, l)         W_K of target layer l   [out, in]
    (seed, cfg, 5, l)         W_V of target layer l
    (seed, cfg, 6, b)         span lengths of context b
    (seed, cfg, 7, l)         bias of K (only when bias_std > 0)
    (seed, cfg, 8, l)         bias of V
    (seed, cfg, 9, l, b)      native target K of the fit (draw_native_target)
    (seed, cfg, 10, l, b)     native target V of the fit

Values are drawn in float32 and then cast round-to-nearest-even to the
storage dtype; bf16 tensors are returned as their uint16 bit patterns.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class ModelShape:
    """KV-cache shape of one model: layers, KV heads, head_dim, RoPE base.

    ``rope_base <= 0`` means the model applies no rotary embedding to K.
    """

    n_layers: int
    n_kv_heads: int
    head_dim: int
    rope_base: float


@dataclass(frozen=True)
class Spec:
    """Everything needed to draw one problem instance."""

    cfg_id: int
    name: str
    src: ModelShape
    tgt: ModelShape
    mix: int                      # source layers concatenated per target layer
    layer_map: tuple              # flat [tgt.n_layers * mix] source layer ids
    dtype: str                    # F32 or BF16 (KV and weights)
    src_tokens: int               # T_s, same for every context
    batch: int = 1
    span_lo: int = 0              # 0 -> identity alignment (same tokenizer)
    span_hi: int = 0
    outliers: int = 0             # channels per (layer, head) scaled by outlier_scale
    outlier_scale: float = 20.0
    w_std: Optional[float] = None  # default 1/sqrt(in)
    bias_std: float = 0.0
    seed: int = 0

    @property
    def d_in(self) -> int:
        return self.mix * self.src.n_kv_heads * self.src.head_dim

    @property
    def d_out(self) -> int:
        return self.tgt.n_kv_heads * self.tgt.head_dim

    @property
    def identity_align(self) -> bool:
        return self.span_lo == 0

    def replace(self, **kw) -> "Spec":
        return dataclasses.replace(self, **kw)


# ---------------------------------------------------------------------------
# Layer maps (integer arithmetic only, no floating point involved)
# ---------------------------------------------------------------------------

def identity_map(n: int) -> tuple:
    return tuple(range(n))


def rounded_ratio_map(lt: int, ls: int) -> tuple:
    """Target layer l reads source layer round(l*(ls-1)/(lt-1)).

    Computed exactly as floor((2*l*(ls-1) + (lt-1)) / (2*(lt-1))), i.e.
    round-half-up on the exact rational; for (lt, ls) = (26, 28) no ties occur.
    """
    num, den = ls - 1, lt - 1
    return tuple((2 * l * num + den) // (2 * den) for l in range(lt))


def window_map(lt: int, ls: int, m: int) -> tuple:
    """Target layer l mixes source layers floor(l*ls/lt) + {0..m-1}."""
    out = []
    for l in range(lt):
        start = (l * ls) // lt
        out.extend(start + j for j in range(m))
    return tuple(out)


# ---------------------------------------------------------------------------
# The five workloads
# ---------------------------------------------------------------------------

QWEN7B = ModelShape(28, 4, 128, 1.0e6)
QWEN1_5B = ModelShape(28, 2, 128, 1.0e6)
GEMMA2B = ModelShape(26, 4, 256, 1.0e4)
LLAMA70B = ModelShape(80, 8, 128, 5.0e5)


def config(cfg_id: int, src_tokens: Optional[int] = None, batch: Optional[int] = None,
           seed: int = 0) -> Spec:
    """The five workloads, by number (1-based).

    1  tiny fp32 smoke: 4 layers, 2x64, base 1e4 on both sides, T=256
    2  Qwen2.5-7B -> Qwen2.5-1.5B, bf16, same tokenizer, T=4096, outliers
    3  Qwen2.5-1.5B -> Gemma-2-2B, bf16, spans of 1-3 tokens, T=4096
    4  config 3 at T in {1K..16K}, batch of 8 contexts
    5  Llama3.1-70B -> Qwen2.5-7B, bf16, 3-layer windows, spans of 1-2, T=8192
    """
    if cfg_id == 1:
        s = ModelShape(4, 2, 64, 1.0e4)
        spec = Spec(1, "tiny-f32", s, s, 1, identity_map(4), F32, 256)
    elif cfg_id == 2:
        spec = Spec(2, "qwen2.5-7b->qwen2.5-1.5b", QWEN7B, QWEN1_5B, 1,
                    identity_map(28), BF16, 4096, outliers=4)
    elif cfg_id == 3:
        spec = Spec(3, "qwen2.5-1.5b->gemma-2-2b", QWEN1_5B, GEMMA2B, 1,
                    rounded_ratio_map(26, 28), BF16, 4096, span_lo=1, span_hi=3)
    elif cfg_id == 4:
        spec = Spec(4, "qwen2.5-1.5b->gemma-2-2b-batched", QWEN1_5B, GEMMA2B, 1,
                    rounded_ratio_map(26, 28), BF16, 4096, batch=8, span_lo=1, span_hi=3)
    elif cfg_id == 5:
        spec = Spec(5, "llama3.1-70b->qwen2.5-7b", LLAMA70B, QWEN7B, 3,
                    window_map(28, 80, 3), BF16, 8192, span_lo=1, span_hi=2, outliers=4)
    else:
        raise ValueError(f"unknown config {cfg_id}")
    kw = {"seed": seed}
    if src_tokens is not None:
        kw["src_tokens"] = int(src_tokens)
    if batch is not None:
        kw["batch"] = int(batch)
    return spec.replace(**kw)


# ---------------------------------------------------------------------------
# dtype helpers (storage casts only)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16, returned as uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if np.isnan(x).any():
        raise ValueError("NaN in synthetic input")
    u = x.view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == BF16:
        return f32_to_bf16_bits(x)
    raise ValueError(dtype)


def storage_to_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return np.asarray(x, dtype=np.float32) if dtype == F32 else bf16_bits_to_f32(x)


# ---------------------------------------------------------------------------
# Problem instance
# ---------------------------------------------------------------------------

@dataclass
class Problem:
    """Host arrays of one problem instance (all C-contiguous).

    src_k, src_v : [Ls, B, Hs, T_s, Ds]   storage dtype
    w_k, w_v     : [Lt, out, in]          storage dtype (nn.Linear order)
    b_k, b_v     : [Lt, out] float32, or None (zero bias)
    tgt_tokens   : [B] int32 (T_t per context)
    row_ptr      : [R+1] int32 or None (identity alignment)
    col_idx      : [nnz] int32 (source token index within the context)
    weight       : [nnz] float32
    """

    spec: Spec
    src_k: np.ndarray
    src_v: np.ndarray
    w_k: np.ndarray
    w_v: np.ndarray
    b_k: Optional[np.ndarray]
    b_v: Optional[np.ndarray]
    tgt_tokens: np.ndarray
    row_ptr: Optional[np.ndarray]
    col_idx: Optional[np.ndarray]
    weight: Optional[np.ndarray]
    layer_map: np.ndarray = field(default=None)

    @property
    def n_rows(self) -> int:
        return int(self.tgt_tokens.sum())

    @property
    def tgt_capacity(self) -> int:
        return int(self.tgt_tokens.max()) if len(self.tgt_tokens) else 0

    def row_offsets(self) -> np.ndarray:
        off = np.zeros(len(self.tgt_tokens) + 1, dtype=np.int64)
        np.cumsum(self.tgt_tokens, out=off[1:])
        return off


def _rng(spec: Spec, *stream) -> np.random.Generator:
    return np.random.default_rng([spec.seed, spec.cfg_id, *stream])


def draw_spans(spec: Spec, b: int) -> np.ndarray:
    """Span lengths of context b: i.i.d. uniform in [span_lo, span_hi], drawn
    left to right; the last span is truncated so the spans partition [0, T_s)."""
    T = spec.src_tokens
    if T == 0:
        return np.zeros(0, dtype=np.int64)
    lens = _rng(spec, 6, b).integers(spec.span_lo, spec.span_hi + 1, size=T)
    ends = np.cumsum(lens)
    n = int(np.searchsorted(ends, T)) + 1
    lens = lens[:n].copy()
    lens[-1] -= int(ends[n - 1]) - T
    assert lens.sum() == T and lens.min() >= 1
    return lens


def span_csr(spec: Spec):
    """CSR alignment of all contexts: rows concatenated per context.

    Returns (tgt_tokens[B], row_ptr[R+1], col_idx[nnz], weight[nnz]) where row r
    of context b pools source tokens of one span with equal weights
    float32(1/len)."""
    counts, rps, cols, ws = [], [], [], []
    base = 0
    for b in range(spec.batch):
        lens = draw_spans(spec, b)
        counts.append(len(lens))
        rps.append(base + np.cumsum(lens))
        cols.append(np.arange(spec.src_tokens, dtype=np.int32))
        ws.append(np.repeat((1.0 / lens).astype(np.float32), lens))
        base += spec.src_tokens
    row_ptr = np.concatenate([[0]] + rps).astype(np.int32)
    return (np.asarray(counts, dtype=np.int32), row_ptr,
            np.concatenate(cols).astype(np.int32), np.concatenate(ws).astype(np.float32))


def draw_source(spec: Spec, which: int, layers=None) -> np.ndarray:
    """Source K (which=0) or V (which=1) in float32, [Ls, B, Hs, T, Ds].

    ``layers`` restricts the draw to a subset of source layers (others are
    zero); the values of the drawn layers do not depend on the subset."""
    s = spec.src
    out = np.zeros((s.n_layers, spec.batch, s.n_kv_heads, spec.src_tokens, s.head_dim),
                   dtype=np.float32)
    todo = range(s.n_layers) if layers is None else sorted(set(int(x) for x in layers))
    for ls in todo:
        for b in range(spec.batch):
            out[ls, b] = _rng(spec, which, ls, b).standard_normal(
                (s.n_kv_heads, spec.src_tokens, s.head_dim), dtype=np.float32)
        if spec.outliers:
            marks = _outlier_marks(spec, which, ls)
            for h in range(s.n_kv_heads):
                out[ls, :, h, :, marks[h]] *= np.float32(spec.outlier_scale)
    return out


def _outlier_marks(spec: Spec, which: int, ls: int) -> np.ndarray:
    """Outlier channels of source layer ``ls``: bool [Hs, Ds]."""
    s = spec.src
    marks = np.zeros((s.n_kv_heads, s.head_dim), dtype=bool)
    if spec.outliers:
        r = _rng(spec, 2 + which, ls)
        for h in range(s.n_kv_heads):
            marks[h, r.choice(s.head_dim, size=spec.outliers, replace=False)] = True
    return marks


def outlier_channels(spec: Spec, which: int) -> np.ndarray:
    """The channels that draw_source scales, K (which=0) or V (which=1):
    bool [Ls, Hs, Ds] (all False without outliers)."""
    return np.stack([_outlier_marks(spec, which, ls) for ls in range(spec.src.n_layers)])


def draw_weights(spec: Spec, which: int) -> np.ndarray:
    """W_K (which=0) or W_V (which=1), float32 [Lt, out, in] ~ N(0, w_std^2)."""
    std = spec.w_std if spec.w_std is not None else 1.0 / np.sqrt(spec.d_in)
    w = np.empty((spec.tgt.n_layers, spec.d_out, spec.d_in), dtype=np.float32)
    for l in range(spec.tgt.n_layers):
        w[l] = _rng(spec, 4 + which, l).standard_normal((spec.d_out, spec.d_in),
                                                          dtype=np.float32) * np.float32(std)
    return w


def draw_bias(spec: Spec, which: int) -> Optional[np.ndarray]:
    if spec.bias_std <= 0:
        return None
    b = np.empty((spec.tgt.n_layers, spec.d_out), dtype=np.float32)
    for l in range(spec.tgt.n_layers):
        b[l] = _rng(spec, 7 + which, l).standard_normal(spec.d_out, dtype=np.float32) \
            * np.float32(spec.bias_std)
    return b


def make_problem(spec: Spec, src_layers=None) -> Problem:
    """Draw one full problem instance of ``spec`` (see module docstring)."""
    assert len(spec.layer_map) == spec.tgt.n_layers * spec.mix
    src_k = to_storage(draw_source(spec, 0, src_layers), spec.dtype)
    src_v = to_storage(draw_source(spec, 1, src_layers), spec.dtype)
    w_k = to_storage(draw_weights(spec, 0), spec.dtype)
    w_v = to_storage(draw_weights(spec, 1), spec.dtype)
    if spec.identity_align:
        tgt_tokens = np.full(spec.batch, spec.src_tokens, dtype=np.int32)
        row_ptr = col_idx = weight = None
    else:
        tgt_tokens, row_ptr, col_idx, weight = span_csr(spec)
    return Problem(spec, src_k, src_v, w_k, w_v, draw_bias(spec, 0), draw_bias(spec, 1),
                   tgt_tokens, row_ptr, col_idx, weight,
                   np.asarray(spec.layer_map, dtype=np.int32))


def draw_native_target(spec: Spec, which: int, tgt_tokens) -> np.ndarray:
    """Stand-in for a target model's own prefill cache, K (which=0) or V
    (which=1): N(0, 1) rows [Lt, B, Ht, cap, Dt] in the storage dtype, rows
    past a context's T_t zero.  Streams (seed, cfg, 9 + which, l, b)."""
    t = spec.tgt
    tt = np.asarray(tgt_tokens)
    cap = int(tt.max()) if len(tt) else 0
    out = np.zeros((t.n_layers, spec.batch, t.n_kv_heads, cap, t.head_dim), dtype=np.float32)
    for l in range(t.n_layers):
        for b in range(spec.batch):
            n = int(tt[b])
            out[l, b, :, :n] = _rng(spec, 9 + which, l, b).standard_normal(
                (t.n_kv_heads, n, t.head_dim), dtype=np.float32)
    return to_storage(out, spec.dtype)


def draw_lowrank(spec: Spec, rank: int):
    """Low-rank translator factors (u_k, v_k, u_v, v_v) in the storage dtype:
    U [Lt, out, r] ~ N(0, 1/r), V [Lt, r, in] ~ N(0, 1/in), so that U V z has
    the scale of the dense draw.  Streams (seed, cfg, 11 + which, l, 0 | 1)."""
    out = []
    for which in (0, 1):
        u = np.empty((spec.tgt.n_layers, spec.d_out, rank), dtype=np.float32)
        v = np.empty((spec.tgt.n_layers, rank, spec.d_in), dtype=np.float32)
        for l in range(spec.tgt.n_layers):
            u[l] = _rng(spec, 11 + which, l, 0).standard_normal(
                (spec.d_out, rank), dtype=np.float32) * np.float32(1.0 / np.sqrt(rank))
            v[l] = _rng(spec, 11 + which, l, 1).standard_normal(
                (rank, spec.d_in), dtype=np.float32) * np.float32(1.0 / np.sqrt(spec.d_in))
        out += [to_storage(u, spec.dtype), to_storage(v, spec.dtype)]
    return tuple(out)


def draw_mixture(spec: Spec, n_mix: int, with_bias: bool = True):
    """A mixture of ``n_mix`` translators: alpha [K] float64 ~ Dirichlet(1)
    (stream 15), members w_k, w_v [K, Lt, out, in] ~ N(0, 1/in) in the
    storage dtype (streams 13 + which, k, l) and biases b_k, b_v fp32
    [K, Lt, out] ~ N(0, bias_std^2) (streams 17 + which, k, l) or None.
    Returns (alpha, w_k, w_v, b_k, b_v)."""
    alpha = _rng(spec, 15).dirichlet(np.ones(n_mix))
    std = np.float32(1.0 / np.sqrt(spec.d_in))
    ws, bs = [], []
    for which in (0, 1):
        w = np.empty((n_mix, spec.tgt.n_layers, spec.d_out, spec.d_in), dtype=np.float32)
        b = np.empty((n_mix, spec.tgt.n_layers, spec.d_out), dtype=np.float32)
        for k in range(n_mix):
            for l in range(spec.tgt.n_layers):
                w[k, l] = _rng(spec, 13 + which, k, l).standard_normal(
                    (spec.d_out, spec.d_in), dtype=np.float32) * std
                b[k, l] = _rng(spec, 17 + which, k, l).standard_normal(
                    spec.d_out, dtype=np.float32) * np.float32(spec.bias_std)
        ws.append(to_storage(w, spec.dtype))
        bs.append(b if with_bias else None)
    return alpha, ws[0], ws[1], bs[0], bs[1]


def llama31_inv_freq(base: float, head_dim: int, factor: float = 8.0, low: float = 1.0,
                     high: float = 4.0, original_context: int = 8192) -> np.ndarray:
    """RoPE frequencies with the long-context rescaling published with
    Llama 3.1 (an input table for the ``inv_freq`` override): components
    whose wavelength 2 pi / theta is below original_context / high keep their
    frequency, those above original_context / low are slowed by ``factor``,
    and the band in between blends the two linearly in
    original_context / wavelength."""
    out = np.array([base ** (-2.0 * i / head_dim) for i in range(head_dim // 2)])
    for i, th in enumerate(out):
        wavelen = 2.0 * np.pi / th
        if wavelen < original_context / high:
            continue
        if wavelen > original_context / low:
            out[i] = th / factor
            continue
        s = (original_context / wavelen - low) / (high - low)
        out[i] = (1.0 - s) * th / factor + s * th
    return out


def tiny_spec(**kw) -> Spec:
    """A small custom problem for property tests; every field overridable."""
    base = dict(cfg_id=100, name="tiny", src=ModelShape(3, 2, 8, 1.0e4),
                tgt=ModelShape(2, 3, 4, 500.0), mix=1, layer_map=(2, 0), dtype=F32,
                src_tokens=9, batch=2)
    base.update(kw)
    return Spec(**base)
