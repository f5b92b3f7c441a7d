"""The translator-variant oracle (oracle/variants.py) against the dense
translation oracle, which is pinned independently (tests/oracle_pins.py).

* Low rank with U = I and V = W is the dense translator.
* Low rank with small-integer U, V (so U V is exact in float32) equals the
  dense oracle run with W = U V.
* A one-member mixture with weight 1 is the dense translator; a two-member
  mixture with dyadic weights and small-integer members equals the dense
  oracle with the weighted sum of weights and biases (exact in float32).
* Planted mistakes in a copy of the variant oracle each fail a pin.
"""
import dataclasses
import importlib.util
import os

import numpy as np
import pytest

from oracle import oracle as O
from oracle import variants as V
from paper_2608_30963_amd import synth as S


def _spec(**kw):
    base = dict(cfg_id=500, name="variants", src=S.ModelShape(3, 2, 16, 1.0e4),
                tgt=S.ModelShape(2, 2, 8, 1.0e6), mix=2, layer_map=(0, 2, 1, 2), dtype=S.F32,
                src_tokens=40, batch=2, span_lo=1, span_hi=2, bias_std=0.5, seed=7)
    base.update(kw)
    return S.Spec(**base)


def _ints(rng, shape, lo=-2, hi=3):
    return rng.integers(lo, hi, size=shape).astype(np.float32)


def _close(a, b, tol=1e-9):
    m = ~np.isnan(b)
    assert np.array_equal(np.isnan(a), np.isnan(b))
    assert np.max(np.abs(a[m] - b[m])) <= tol * max(1.0, np.max(np.abs(b[m])))


def _pins(mod):
    rng = np.random.default_rng(3)
    prob = S.make_problem(_spec())
    spec = prob.spec
    Lt, dout, din = spec.tgt.n_layers, spec.d_out, spec.d_in
    dk, dv = O.translate(prob)
    # low rank, U = I, V = W
    eye = np.stack([np.eye(dout, dtype=np.float32)] * Lt)
    lk, lv = mod.translate_lowrank(prob, eye, prob.w_k, eye, prob.w_v, prob.b_k, prob.b_v)
    _close(lk, dk)
    _close(lv, dv)
    # low rank with integer factors
    r = 3
    uk, vk = _ints(rng, (Lt, dout, r)), _ints(rng, (Lt, r, din))
    uv, vv = _ints(rng, (Lt, dout, r)), _ints(rng, (Lt, r, din))
    dense = dataclasses.replace(prob, w_k=np.einsum("lor,lri->loi", uk, vk).astype(np.float32),
                                w_v=np.einsum("lor,lri->loi", uv, vv).astype(np.float32))
    rk, rv = O.translate(dense)
    lk, lv = mod.translate_lowrank(prob, uk, vk, uv, vv, prob.b_k, prob.b_v)
    _close(lk, rk)
    _close(lv, rv)
    # mixture: one member, weight 1
    mk, mv = mod.translate_mixture(prob, [1.0], prob.w_k[None], prob.w_v[None],
                                   prob.b_k[None], prob.b_v[None])
    _close(mk, dk)
    _close(mv, dv)
    # mixture: two integer members, dyadic weights
    alpha = [0.25, 0.75]
    wk = _ints(rng, (2, Lt, dout, din))
    wv = _ints(rng, (2, Lt, dout, din))
    bk = _ints(rng, (2, Lt, dout))
    bv = _ints(rng, (2, Lt, dout))
    comb = dataclasses.replace(
        prob, w_k=(0.25 * wk[0] + 0.75 * wk[1]).astype(np.float32),
        w_v=(0.25 * wv[0] + 0.75 * wv[1]).astype(np.float32),
        b_k=(0.25 * bk[0] + 0.75 * bk[1]).astype(np.float32),
        b_v=(0.25 * bv[0] + 0.75 * bv[1]).astype(np.float32))
    ck, cv = O.translate(comb)
    mk, mv = mod.translate_mixture(prob, alpha, wk, wv, bk, bv)
    _close(mk, ck)
    _close(mv, cv)


def test_variant_pins():
    _pins(V)


MUTANTS = {
    "latent_skips_v": ("latent = Z @ V[l].T", "latent = Z[:, :V[l].shape[0]]"),
    "u_not_transposed": ("u = latent @ U[l].T", "u = latent @ U[l].reshape(U[l].shape[1], -1)"),
    "mixture_ignores_alpha": ("u += alpha[k] * uk", "u += uk"),
    "mixture_bias_unweighted": ("uk = uk + np.asarray(b[k, l], dtype=np.float64)", "pass"),
    "target_rope_sign": ("y = F.rotate(y, np.arange(n), theta, +1.0)",
                         "y = F.rotate(y, np.arange(n), theta, -1.0)"),
    "lowrank_bias_dropped": ("u = u + np.asarray(b[l], dtype=np.float64)", "pass"),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_variant_mutant_fails(name, tmp_path):
    src = open(V.__file__).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    path = os.path.join(tmp_path, f"variants_{name}.py")
    open(path, "w").write(src.replace(a, b))
    spec = importlib.util.spec_from_file_location(f"variants_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    with pytest.raises((AssertionError, ValueError)):
        _pins(mod)
