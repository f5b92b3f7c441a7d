"""GPU parity of boundary options the five workloads do not exercise, against
the fp64 oracle element by element, and of the validation mode:

* RoPE off on one side only (rope_base 0: a model without rotary
  embeddings, Section 4's models that differ in attention configuration);
* frequency override tables (the Llama 3.1 rescaled frequencies that a real
  Llama-3.1 cache carries; an arbitrary table on the target side);
* shapes the matrix-core kernel does not tile (head_dim 80, a target
  head_dim of 576), which run the general kernel on bf16 data;
* KVX_VALIDATE=1 rejecting device CSRs that break the alignment contract,
  with nothing enqueued.
"""
import dataclasses
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _full(prob, expect_kernel, src_inv_freq=None, tgt_inv_freq=None,
          precision=kvx.KVX_PREC_BF16X2):
    spec = prob.spec
    print(f"[options] {spec.name} src base {spec.src.rope_base} tgt base {spec.tgt.rope_base} "
          f"tables {src_inv_freq is not None}/{tgt_inv_freq is not None}", flush=True)
    dev = U.DevProblem(prob, precision, src_inv_freq=src_inv_freq, tgt_inv_freq=tgt_inv_freq)
    assert dev.tr.info().kernel == expect_kernel
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap, src_inv_freq=src_inv_freq,
                         tgt_inv_freq=tgt_inv_freq)
    m = U.check_full(dev, rk, rv, spec.name, 0.75)  # the split mode's bound (test_parity_gpu)
    U.summarize(m, spec.name)
    dev.close()


def _side(spec, src_base=None, tgt_base=None):
    src = spec.src if src_base is None else dataclasses.replace(spec.src, rope_base=src_base)
    tgt = spec.tgt if tgt_base is None else dataclasses.replace(spec.tgt, rope_base=tgt_base)
    return spec.replace(src=src, tgt=tgt)


def test_source_without_rope():
    spec = _side(S.config(2, src_tokens=300), src_base=0.0).replace(name="no-src-rope")
    _full(S.make_problem(spec), 1)


def test_target_without_rope():
    spec = _side(S.config(3, src_tokens=700, batch=2), tgt_base=0.0).replace(name="no-tgt-rope")
    _full(S.make_problem(spec), 1)


def test_llama31_rescaled_source_frequencies():
    """Source frequencies of a Llama-3.1 cache (rescaled table), 3-layer
    windows, spans; 8K positions so the rescaled low frequencies matter."""
    spec = S.config(5, src_tokens=384)
    prob = S.make_problem(spec)
    _full(prob, 1, src_inv_freq=S.llama31_inv_freq(spec.src.rope_base, spec.src.head_dim))


def test_tables_on_both_sides_long_context():
    """Tables on both sides (the target's arbitrary) at 8K source tokens, where
    position times frequency is largest."""
    spec = S.config(3, src_tokens=8192)
    rng = np.random.default_rng(3)
    tgt_tab = np.sort(rng.uniform(1e-5, 1.0, spec.tgt.head_dim // 2))[::-1].copy()
    src_tab = S.llama31_inv_freq(spec.src.rope_base, spec.src.head_dim)
    prob = S.make_problem(spec)
    _full(prob, 1, src_inv_freq=src_tab, tgt_inv_freq=tgt_tab)


def test_table_with_zero_base():
    """A table switches RoPE on for a side whose base is 0."""
    spec = _side(S.config(2, src_tokens=200), src_base=0.0, tgt_base=0.0).replace(name="zero-base")
    prob = S.make_problem(spec)
    _full(prob, 1, src_inv_freq=S.llama31_inv_freq(5.0e5, 128),
          tgt_inv_freq=S.llama31_inv_freq(1.0e6, 128))


HD80 = S.ModelShape(3, 8, 80, 1.0e4)


def test_bf16_general_kernel_head_dim_80():
    """head_dim 80 on both sides (din 640, dout 320): the target head is not a
    multiple of 64, so the plan runs the general kernel on bf16 data."""
    spec = S.Spec(301, "hd80", HD80, S.ModelShape(2, 4, 80, 5.0e5), 1, (2, 0), S.BF16, 300,
                  batch=2, span_lo=1, span_hi=3, bias_std=0.2)
    _full(S.make_problem(spec), 0)


def test_bf16_wide_target_head_runs_general_kernel():
    """A target head_dim of 576 (above the matrix-core kernel's 512) is
    planned on the general kernel and translated correctly."""
    spec = S.Spec(302, "tgt576", S.ModelShape(2, 2, 128, 1.0e6), S.ModelShape(2, 1, 576, 1.0e4),
                  1, (1, 0), S.BF16, 200)
    _full(S.make_problem(spec), 0)


# ---------------------------------------------------------------------------
# Validation mode
# ---------------------------------------------------------------------------

@pytest.fixture
def validate_env():
    old = os.environ.get("KVX_VALIDATE")
    os.environ["KVX_VALIDATE"] = "1"
    yield
    if old is None:
        del os.environ["KVX_VALIDATE"]
    else:
        os.environ["KVX_VALIDATE"] = old


def _bad_csrs(prob):
    """(name, row_ptr, col_idx, weight) variants that break the contract."""
    rp, ci, w = prob.row_ptr.copy(), prob.col_idx.copy(), prob.weight.copy()
    out = []
    r = rp.copy()
    r[5], r[6] = r[6], r[5]                       # not monotone
    out.append(("non-monotone", r, ci, w))
    r = rp.copy()
    r[0] = 1                                      # row_ptr[0] != 0
    out.append(("nonzero-start", r, ci, w))
    c = ci.copy()
    c[7] = prob.spec.src_tokens                   # past the context
    out.append(("col-past-end", rp, c, w))
    c = ci.copy()
    c[3] = -1
    out.append(("col-negative", rp, c, w))
    # an empty row: merge row 9's entries into row 8
    r = np.delete(rp, 9)
    r = np.insert(r, 9, r[8])
    out.append(("empty-row", r, ci, w))
    ww = w.copy()
    ww[prob.row_ptr[4]] *= np.float32(1.5)        # row 4 no longer sums to 1
    out.append(("row-sum", rp, ci, ww))
    return out


def test_validate_rejects_bad_csr(validate_env):
    spec = S.config(3, src_tokens=300, batch=2)
    prob = S.make_problem(spec)
    dev = U.DevProblem(prob)
    T = U.torch()
    dev.run()  # the drawn map passes validation
    T.cuda.synchronize()
    assert not T.isnan(dev.tgt_k[:, :, :, :int(prob.tgt_tokens.min())]).any()
    for name, rp, ci, w in _bad_csrs(prob):
        print(f"[validate] {name}", flush=True)
        dev.tgt_k.fill_(float("nan"))
        dev.tgt_v.fill_(float("nan"))
        d_rp, d_ci, d_w = U.np_to_dev(rp, S.F32), U.np_to_dev(ci, S.F32), U.np_to_dev(w, S.F32)
        io, keep = kvx.make_io(spec.batch, spec.src_tokens, dev.src_k, dev.src_v, dev.tgt_k,
                               dev.tgt_v, dev.cap, prob.tgt_tokens, d_rp, d_ci, d_w)
        st = kvx.kvx_translate_status(dev.tr.plan, io,
                                      T.cuda.current_stream().cuda_stream)
        T.cuda.synchronize()
        assert st == kvx.KVX_EDATA, (name, st)
        assert T.isnan(dev.tgt_k).all() and T.isnan(dev.tgt_v).all(), \
            f"{name}: a rejected call wrote the target"
        del keep
    dev.close()


def test_validate_accepts_fp32_one_third_weights(validate_env):
    """Rows of three entries weigh float32(1/3) each: their sum is 1 + 3e-8,
    inside the bound n * 2^-23."""
    spec = S.config(3, src_tokens=600)
    prob = S.make_problem(spec)
    lens = np.diff(prob.row_ptr)
    assert (lens == 3).any()
    dev = U.DevProblem(prob)
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    U.check_full(dev, rk, rv, "validated")
    dev.close()
