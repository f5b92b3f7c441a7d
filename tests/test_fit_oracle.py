"""The fit oracle (oracle/fit.py) against facts outside itself.

* Recovery: native target caches produced by the (independently pinned)
  translation oracle from known weights W*, b* are fitted back to W*, b*
  exactly (lam = 0, fp64 targets) -- for identity and span alignment, layer
  mixing, and RoPE on both sides.  A sign, pairing, position, pooling,
  layer-map or orientation slip anywhere in the fit breaks this.
* The pre-rotation objective the fit minimises equals the squared distance
  between the translated cache (translation oracle, fitted weights) and the
  native cache: the Section 5 objective with D = squared Frobenius distance.
* Optimality: the fitted weights beat random perturbations, a one feature
  regression without RoPE matches its hand-derived closed form, and the
  unpenalised bias satisfies b = mean(Y) - W mean(Z).
* Limits: lam -> infinity drives W to 0 and b to the mean target row.
"""
import dataclasses

import numpy as np
import pytest

from oracle import fit as F
from oracle import oracle as O
from paper_2608_30963_amd import synth as S


def _spec(**kw):
    base = dict(cfg_id=300, name="fit-pin", src=S.ModelShape(3, 2, 32, 1.0e4),
                tgt=S.ModelShape(2, 2, 16, 1.0e6), mix=1, layer_map=(2, 0), dtype=S.F32,
                src_tokens=150, batch=2, bias_std=0.3, seed=3)
    base.update(kw)
    return S.Spec(**base)


SPECS = {
    "identity": _spec(),
    "spans-mix2": _spec(mix=2, layer_map=(0, 1, 2, 1), src_tokens=420, span_lo=1, span_hi=3,
                        batch=1),
    "bf16-outliers": _spec(dtype=S.BF16, outliers=2, src_tokens=200),
}


def _native(prob):
    """Target caches from the translation oracle (fp64)."""
    return O.translate(prob)


@pytest.mark.parametrize("name", list(SPECS))
def test_recovery_exact(name):
    prob = S.make_problem(SPECS[name])
    tk, tv = _native(prob)
    wk, wv, bk, bv = F.fit(prob, tk, tv, lam=0.0, fit_bias=True)
    for got, ref in ((wk, prob.w_k), (wv, prob.w_v)):
        ref = F._widen(ref)
        assert np.max(np.abs(got - ref)) <= 1e-9 * np.max(np.abs(ref)), name
    for got, ref in ((bk, prob.b_k), (bv, prob.b_v)):
        assert np.max(np.abs(got - ref.astype(np.float64))) <= 1e-9, name


def test_objective_is_cache_distance():
    """||translate(W, b) - native||^2 over the valid rows (translation oracle)
    equals the fit's pre-rotation data term for the same W, b."""
    spec = _spec(src_tokens=90)
    prob = S.make_problem(spec)
    tk, tv = _native(prob)
    rng = np.random.default_rng(0)
    tk_noisy = tk + 0.05 * rng.standard_normal(tk.shape)
    tv_noisy = tv + 0.05 * rng.standard_normal(tv.shape)
    wk, wv, bk, bv = F.fit(prob, tk_noisy, tv_noisy, lam=0.5, fit_bias=True)
    fitted = dataclasses.replace(prob, w_k=wk.astype(np.float32), w_v=wv.astype(np.float32),
                                 b_k=bk.astype(np.float32), b_v=bv.astype(np.float32))
    ok, ov = O.translate(fitted)
    for which, native, trans, W, b in ((0, tk_noisy, ok, wk, bk), (1, tv_noisy, ov, wv, bv)):
        cache = float(((trans - native) ** 2).sum())      # every row valid (identity)
        W32 = W.astype(np.float32).astype(np.float64)
        b32 = b.astype(np.float32).astype(np.float64)
        data = F.objective(fitted, native, which, W32, b32, lam=0.0)
        assert abs(cache - data) <= 1e-9 * data, (which, cache, data)


def test_fit_beats_perturbations():
    spec = _spec(src_tokens=80)
    prob = S.make_problem(spec)
    tk, tv = _native(prob)
    rng = np.random.default_rng(1)
    tk = tk + 0.1 * rng.standard_normal(tk.shape)
    lam = 2.0
    wk, wv, bk, bv = F.fit(prob, tk, tv, lam=lam, fit_bias=True)
    best = F.objective(prob, tk, 0, wk, bk, lam)
    for _ in range(5):
        dW = 1e-3 * rng.standard_normal(wk.shape)
        db = 1e-3 * rng.standard_normal(bk.shape)
        assert F.objective(prob, tk, 0, wk + dW, bk + db, lam) > best


def test_one_feature_closed_form():
    """din = 1, no RoPE, no bias: w = sum(z y) / (sum(z^2) + lam)."""
    rng = np.random.default_rng(2)
    z = rng.standard_normal((50, 1))
    y = rng.standard_normal((50, 3))
    lam = 0.7
    W, b = F.solve(z, y, lam, fit_bias=False)
    ref = (z[:, 0] @ y) / (z[:, 0] @ z[:, 0] + lam)
    assert b is None
    assert np.allclose(W[:, 0], ref, rtol=1e-12, atol=0)


def test_bias_centering():
    """With an unpenalised bias, d/db = 0 gives b = mean(Y) - W mean(Z)."""
    rng = np.random.default_rng(9)
    Z = rng.standard_normal((40, 3)) + 2.0
    Y = rng.standard_normal((40, 5)) - 1.0
    W, b = F.solve(Z, Y, 1.0, True)
    assert np.allclose(b, Y.mean(axis=0) - W @ Z.mean(axis=0), rtol=0, atol=1e-12)


def test_huge_ridge_limit():
    spec = _spec(src_tokens=60)
    prob = S.make_problem(spec)
    tk, tv = _native(prob)
    wk, wv, bk, bv = F.fit(prob, tk, tv, lam=1e14, fit_bias=True)
    assert np.max(np.abs(wk)) < 1e-8 and np.max(np.abs(wv)) < 1e-8
    yk = F.target_rows(prob, tk, 0)
    assert np.allclose(bk, yk.mean(axis=1), atol=1e-6)


def test_rotate_is_rope():
    """The fit's rotation agrees with the translation oracle's RoPE (which is
    pinned to the closed form elsewhere) at arbitrary positions."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((5, 16))
    pos = np.array([0, 1, 7, 300, 4095])
    theta = F.inv_freq(16, 1.0e4)
    y = F.rotate(x, pos, theta, +1.0)
    for i in range(5):
        assert np.allclose(y[i], O.rope(x[i], float(pos[i]), 1.0e4), rtol=0, atol=1e-12)
