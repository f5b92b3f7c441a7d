"""Planted mistakes in a copy of the fit oracle must each fail a fit pin.

Each mutant is a textual edit of ``oracle/fit.py`` loaded as a separate
module on the CPU; the recovery and cache-distance pins of
``test_fit_oracle.py`` run against it.  A mutant that passes every pin
would mean the pins cannot see that class of mistake.
"""
import importlib.util
import os

import numpy as np
import pytest

from oracle import fit as F
from oracle import oracle as O
from paper_2608_30963_amd import synth as S

MUTANTS = {
    "source_derotate_sign": ("x = rotate(x, np.arange(T), theta, -1.0)",
                             "x = rotate(x, np.arange(T), theta, +1.0)"),
    "target_not_derotated": ("y = rotate(y, np.arange(n), theta, -1.0)", "pass"),
    "target_derotate_sign": ("y = rotate(y, np.arange(n), theta, -1.0)",
                             "y = rotate(y, np.arange(n), theta, +1.0)"),
    "rotation_sign": ("x1 * c - x2 * s, x2 * c + x1 * s", "x1 * c + x2 * s, x2 * c - x1 * s"),
    "freq_exponent": ("base ** (-2.0 * i / head_dim)", "base ** (-i / head_dim)"),
    "pool_weight_ignored": ("zb[t] += float(prob.weight[e]) * xb[int(prob.col_idx[e])]",
                            "zb[t] += xb[int(prob.col_idx[e])]"),
    "mix_layer_ignored": ("ls = int(lmap[layer * spec.mix + j])",
                          "ls = int(lmap[layer * spec.mix])"),
    "bias_penalised": ("D[-1] = 0.0", "D[-1] = 1.0"),
    "w_not_transposed": ("W = X[:din].T.copy()", "W = X[:din].reshape(X.shape[1], din).copy()"),
    "v_rotated": ("use_rope = which == 0 and s.rope_base > 0", "use_rope = s.rope_base > 0"),
}


def _load_mutant(name, tmp_path):
    src = open(F.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    path = os.path.join(tmp_path, f"fit_{name}.py")
    open(path, "w").write(src.replace(a, b))
    spec = importlib.util.spec_from_file_location(f"fit_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _pins_pass(mod) -> bool:
    cases = [
        S.Spec(300, "m1", S.ModelShape(3, 2, 32, 1.0e4), S.ModelShape(2, 2, 16, 1.0e6), 1, (2, 0),
               S.F32, 150, batch=2, bias_std=0.3, seed=3),
        S.Spec(300, "m2", S.ModelShape(3, 2, 32, 1.0e4), S.ModelShape(2, 2, 16, 1.0e6), 2,
               (0, 1, 2, 1), S.F32, 420, span_lo=1, span_hi=3, bias_std=0.3, seed=3),
    ]
    for spec in cases:
        prob = S.make_problem(spec)
        tk, tv = O.translate(prob)
        try:
            wk, wv, bk, bv = mod.fit(prob, tk, tv, lam=0.0, fit_bias=True)
        except Exception:
            return False
        for got, ref in ((wk, prob.w_k), (wv, prob.w_v), (bk, prob.b_k), (bv, prob.b_v)):
            ref = np.asarray(ref, dtype=np.float64)
            if got.shape != ref.shape or not np.allclose(got, ref, rtol=0, atol=1e-8):
                return False
    # ridge with an unpenalised bias: b = mean(Y) - W mean(Z) (set d/db = 0)
    rng = np.random.default_rng(9)
    Z = rng.standard_normal((40, 3)) + 2.0
    Y = rng.standard_normal((40, 3)) - 1.0
    try:
        W, b = mod.solve(Z, Y, 1.0, True)
    except Exception:
        return False
    return np.allclose(b, Y.mean(axis=0) - W @ Z.mean(axis=0), rtol=0, atol=1e-12)


def test_unmutated_passes(tmp_path):
    assert _pins_pass(F)


@pytest.mark.parametrize("name", list(MUTANTS))
def test_mutant_fails(name, tmp_path):
    assert not _pins_pass(_load_mutant(name, tmp_path)), f"mutant {name} passed every pin"
