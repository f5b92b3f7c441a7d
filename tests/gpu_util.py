"""Helpers of the GPU tests: upload a problem, run the library, compare with
the oracle.

Tolerances (translated K/V against the fp64 oracle, per tensor = one target
layer's K or V):
* bf16: element-wise |g - r| <= 2e-2 * max(1, |r|) and relative Frobenius
  error <= 1e-2.  The literal max-abs bound cannot hold for bf16 outputs above
  |r| = 8 (half an ulp there is 2^-5 > 2e-2), so it scales with |r| beyond 1.
  A tighter guard in bf16 ulps (``ulp_bound``) catches accuracy regressions
  well inside that envelope.
* fp32: the literal bounds, |g - r| <= 1e-5 element-wise and relative
  Frobenius error <= 1e-5.
Integer work (layer map, layer mixing, alignment, head/token indexing) is
checked bit-exact by ``test_probes_gpu.py``.
"""
from __future__ import annotations

import numpy as np

from paper_2608_30963_amd import kvx, synth as S

TOL = {S.BF16: (2e-2, 1e-2), S.F32: (1e-5, 1e-5)}


def torch():
    import torch as _t
    return _t


def np_to_dev(a: np.ndarray, dtype: str):
    T = torch()
    if a is None:
        return None
    if dtype == S.BF16 and a.dtype == np.uint16:
        return T.from_numpy(a.view(np.int16).copy()).view(T.bfloat16).cuda()
    return T.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_to_f64(t, dtype: str) -> np.ndarray:
    T = torch()
    if t.dtype == T.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


class DevProblem:
    """Device copies of a problem's arrays plus a plan."""

    def __init__(self, prob: S.Problem, precision=kvx.KVX_PREC_BF16X2, cap=None, fill=None,
                 lowrank=None, mixture=None, outliers=None, src_inv_freq=None,
                 tgt_inv_freq=None):
        """``lowrank=(u_k, v_k, u_v, v_v)`` or ``mixture=(alpha, w_k, w_v, b_k,
        b_v)`` (host arrays in the storage dtype, biases fp32) build the plan
        from translator factors instead of the problem's dense weights;
        ``outliers=(marks_k, marks_v)`` are the source outlier channels of
        precision KVX_PREC_BF16X2_OUTLIER; ``src_inv_freq`` / ``tgt_inv_freq``
        override the RoPE frequencies of a side."""
        T = torch()
        spec = prob.spec
        self.prob = prob
        self.spec = spec
        dt = spec.dtype
        self.kdtype = kvx.KVX_BF16 if dt == S.BF16 else kvx.KVX_F32
        self.src_k = np_to_dev(prob.src_k, dt)
        self.src_v = np_to_dev(prob.src_v, dt)
        self.w_k = np_to_dev(prob.w_k, dt)
        self.w_v = np_to_dev(prob.w_v, dt)
        self.b_k = np_to_dev(prob.b_k, S.F32)
        self.b_v = np_to_dev(prob.b_v, S.F32)
        self.row_ptr = np_to_dev(prob.row_ptr, S.F32) if prob.row_ptr is not None else None
        self.col_idx = np_to_dev(prob.col_idx, S.F32) if prob.col_idx is not None else None
        self.weight = np_to_dev(prob.weight, S.F32) if prob.weight is not None else None
        self.factors = None
        if lowrank is not None:
            self.factors = tuple(np_to_dev(a, dt) for a in lowrank)
            kw = {"lowrank": self.factors}
        elif mixture is not None:
            alpha, mw_k, mw_v, mb_k, mb_v = mixture
            self.factors = (np_to_dev(mw_k, dt), np_to_dev(mw_v, dt), np_to_dev(mb_k, S.F32),
                            np_to_dev(mb_v, S.F32))
            kw = {"mixture": (list(alpha),) + self.factors}
        else:
            kw = {"w_k": self.w_k, "w_v": self.w_v}
        if outliers is not None:
            kw["outlier_k"], kw["outlier_v"] = outliers
        self.tr = kvx.Translator(spec.src, spec.tgt, spec.mix, spec.layer_map, self.kdtype,
                                 b_k=self.b_k, b_v=self.b_v, precision=precision,
                                 src_inv_freq=src_inv_freq, tgt_inv_freq=tgt_inv_freq, **kw)
        self.cap = prob.tgt_capacity if cap is None else cap
        shape = (spec.tgt.n_layers, spec.batch, spec.tgt.n_kv_heads, self.cap,
                 spec.tgt.head_dim)
        tdt = T.bfloat16 if dt == S.BF16 else T.float32
        fill = float("nan") if fill is None else fill
        self.tgt_k = T.full(shape, fill, dtype=tdt, device="cuda")
        self.tgt_v = T.full(shape, fill, dtype=tdt, device="cuda")

    def run(self, stream=None):
        ident = self.prob.row_ptr is None
        self.tr(self.src_k, self.src_v, self.tgt_k, self.tgt_v, self.cap,
                None if ident else self.prob.tgt_tokens,
                self.row_ptr, self.col_idx, self.weight, stream=stream)
        return self.tgt_k, self.tgt_v

    def close(self):
        self.tr.close()


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bfloat16 numbers at |x| (8 significant bits; subnormal
    spacing 2^-133 below the smallest normal 2^-126)."""
    ax = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
    return np.exp2(e - 7)


def ulp_metrics(got: np.ndarray, ref: np.ndarray):
    """Worst error in bf16 ulps of the reference value (``ulp``), and the same
    with the ulp taken at max(|r|, rms(r) / 16) (``ulp_floor``): near-zero
    outputs of a long contraction carry an absolute error set by the size of
    its terms, which the floored measure reads on the tensor's own scale."""
    if got.size == 0:
        return 0.0, 0.0
    d = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref * ref)))
    u = float((d / bf16_ulp(ref)).max())
    uf = float((d / bf16_ulp(np.maximum(np.abs(ref), rms / 16))).max())
    return u, uf


def check_close(got: np.ndarray, ref: np.ndarray, dtype: str, what: str, ulp_bound=None):
    """Element-wise and relative-Frobenius check; returns the metrics.

    bf16: ``ulp_bound`` (if given) also bounds the floored ulp error (see
    ulp_metrics).  fp32: the element bound is the literal absolute one."""
    el, fro = TOL[dtype]
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    d = np.abs(got - ref)
    if dtype == S.F32:
        scaled = d
    else:
        scaled = d / np.maximum(1.0, np.abs(ref))
    worst = float(scaled.max()) if d.size else 0.0
    rf = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)) if d.size else 0.0
    assert worst <= el, f"{what}: element error {worst:.3e} > {el} (max abs {d.max():.3e})"
    assert rf <= fro, f"{what}: relative Frobenius {rf:.3e} > {fro}"
    m = {"max_scaled": worst, "max_abs": float(d.max()) if d.size else 0.0, "rel_fro": rf}
    if dtype == S.BF16:
        m["ulp"], m["ulp_floor"] = ulp_metrics(got, ref)
        if ulp_bound is not None:
            assert m["ulp_floor"] <= ulp_bound, \
                f"{what}: {m['ulp_floor']:.3f} bf16 ulps > {ulp_bound}"
    return m


def check_full(dev: DevProblem, ref_k: np.ndarray, ref_v: np.ndarray, what: str,
               ulp_bound=None):
    """Compare every valid row of every target layer against the oracle."""
    spec = dev.spec
    gk = dev_to_f64(dev.tgt_k, spec.dtype)
    gv = dev_to_f64(dev.tgt_v, spec.dtype)
    out = []
    tt = dev.prob.tgt_tokens
    for l in range(spec.tgt.n_layers):
        for name, g, r in (("K", gk, ref_k), ("V", gv, ref_v)):
            gs = np.concatenate([g[l, b, :, :tt[b]].reshape(-1) for b in range(spec.batch)])
            rs = np.concatenate([r[l, b, :, :tt[b]].reshape(-1) for b in range(spec.batch)])
            out.append(check_close(gs, rs, spec.dtype, f"{what} layer {l} {name}", ulp_bound))
    return out


def summarize(metrics, what: str) -> dict:
    """Worst of each metric over a list of check_close results; printed, so
    that a test run reports the literal max-abs and ulp errors it saw."""
    keys = ("max_abs", "max_scaled", "rel_fro", "ulp", "ulp_floor")
    out = {k: max(m[k] for m in metrics) for k in keys if metrics and k in metrics[0]}
    print(f"[accuracy] {what}: " + ", ".join(f"{k} {v:.3e}" for k, v in out.items()),
          flush=True)
    return out
