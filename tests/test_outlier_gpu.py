"""GPU tests of precision KVX_PREC_BF16X2_OUTLIER (channel-wise mixed
precision: only the k-steps that hold a marked source channel take the split
operand).

* No channel marked: every k-step is rounded once, so the outputs equal a
  KVX_PREC_BF16 plan's bit for bit; every channel marked: every k-step is
  split, so they equal a KVX_PREC_BF16X2 plan's bit for bit.
* The synthetic workloads' own outlier channels marked: parity with the
  fp64 oracle at the bf16 tolerance of the dense parity tests (element
  2e-2 * max(1, |r|), Frobenius 1e-2), on identity alignment, spans, and two
  source heads per K-chunk with layer mixing -- while a plain BF16 plan is
  measurably less accurate on the same inputs.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

QWEN_SMALL = S.ModelShape(2, 4, 128, 1.0e6)


def _spec(**kw):
    base = dict(cfg_id=400, name="outlier", src=QWEN_SMALL, tgt=S.ModelShape(2, 2, 128, 1.0e6),
                mix=1, layer_map=(1, 0), dtype=S.BF16, src_tokens=300, batch=2, outliers=4,
                bias_std=0.5, seed=5)
    base.update(kw)
    return S.Spec(**base)


def _marks(spec):
    return S.outlier_channels(spec, 0), S.outlier_channels(spec, 1)


def _run(prob, precision, outliers=None):
    print(f"[outlier] {prob.spec.name} prec={precision}", flush=True)
    dev = U.DevProblem(prob, precision, cap=max(1, int(prob.tgt_tokens.max())), outliers=outliers)
    dev.run()
    U.torch().cuda.synchronize()
    return dev


def _same(a, b):
    T = U.torch()
    assert T.equal(a.view(T.int16), b.view(T.int16))


@pytest.mark.parametrize("spans", [False, True])
def test_no_marks_is_bf16_and_all_marks_is_bf16x2(spans):
    spec = _spec(name=f"outlier-extremes-{spans}", **({"span_lo": 1, "span_hi": 3} if spans else {}))
    prob = S.make_problem(spec)
    shape = (spec.src.n_layers, spec.src.n_kv_heads, spec.src.head_dim)
    none = (np.zeros(shape, bool), np.zeros(shape, bool))
    every = (np.ones(shape, bool), np.ones(shape, bool))
    got = _run(prob, kvx.KVX_PREC_BF16X2_OUTLIER, none)
    info = got.tr.info()
    assert info.kernel == 1 and info.split_ksteps == 0 and info.ksteps > 0
    ref = _run(prob, kvx.KVX_PREC_BF16)
    _same(got.tgt_k, ref.tgt_k)
    _same(got.tgt_v, ref.tgt_v)
    got.close()
    ref.close()
    got = _run(prob, kvx.KVX_PREC_BF16X2_OUTLIER, every)
    info = got.tr.info()
    assert info.split_ksteps == info.ksteps > 0
    ref = _run(prob, kvx.KVX_PREC_BF16X2)
    _same(got.tgt_k, ref.tgt_k)
    _same(got.tgt_v, ref.tgt_v)
    got.close()
    ref.close()


@pytest.mark.parametrize("kw", [
    {},
    {"span_lo": 1, "span_hi": 3},
    {"src": S.ModelShape(4, 2, 64, 1.0e4), "tgt": S.ModelShape(2, 3, 128, 1.0e6), "mix": 2,
     "layer_map": (0, 1, 3, 2), "span_lo": 1, "span_hi": 2},
], ids=["ident", "spans", "ds64-mix2"])
def test_marked_outliers_parity(kw):
    spec = _spec(name="outlier-parity", **kw)
    prob = S.make_problem(spec)
    dev = _run(prob, kvx.KVX_PREC_BF16X2_OUTLIER, _marks(spec))
    info = dev.tr.info()
    frac = info.split_ksteps / info.ksteps
    print(f"[outlier] split k-steps {info.split_ksteps} / {info.ksteps} = {frac:.2f}", flush=True)
    assert 0 < info.split_ksteps < info.ksteps
    rk, rv = O.translate(prob, cap=dev.cap)
    m = U.check_full(dev, rk, rv, spec.name)
    worst = max(x["max_scaled"] for x in m)
    dev.close()
    # the marks matter: single rounding everywhere is less accurate here
    plain = _run(prob, kvx.KVX_PREC_BF16)
    gk = U.dev_to_f64(plain.tgt_k, spec.dtype)
    tt = prob.tgt_tokens
    g = np.concatenate([gk[l, b, :, :tt[b]].ravel() for l in range(spec.tgt.n_layers)
                        for b in range(spec.batch)])
    r = np.concatenate([rk[l, b, :, :tt[b]].ravel() for l in range(spec.tgt.n_layers)
                        for b in range(spec.batch)])
    plain_worst = float((np.abs(g - r) / np.maximum(1.0, np.abs(r))).max())
    print(f"[outlier] worst scaled error: marked {worst:.2e}, plain bf16 {plain_worst:.2e}",
          flush=True)
    assert worst < plain_worst
    plain.close()
