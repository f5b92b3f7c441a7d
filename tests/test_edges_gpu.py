"""GPU parity on edge cases, against the fp64 oracle element by element:
more contexts than one launch takes, empty contexts and empty alignment rows,
a single source token, two source heads per K-chunk with layer mixing, a
partly used output tile, a strided source view, and layouts the fused kernel
must refuse rather than mis-read.
"""
import dataclasses

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

QWEN_SMALL = S.ModelShape(2, 2, 128, 1.0e6)


def _spec(**kw):
    base = dict(cfg_id=200, name="edge", src=QWEN_SMALL, tgt=QWEN_SMALL, mix=1,
                layer_map=(1, 0), dtype=S.BF16, src_tokens=40, batch=1, outliers=2,
                bias_std=0.5)
    base.update(kw)
    return S.Spec(**base)


def _check(prob, precision=kvx.KVX_PREC_BF16X2, expect_kernel=1, expect_order=None):
    print(f"[edges] {prob.spec.name} T={prob.spec.src_tokens} B={prob.spec.batch} "
          f"tt={list(prob.tgt_tokens)[:8]}", flush=True)
    dev = U.DevProblem(prob, precision, cap=max(1, int(prob.tgt_tokens.max())))
    assert dev.tr.info().kernel == expect_kernel
    if expect_order is not None:
        assert dev.tr.info().tile_order == expect_order
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    U.check_full(dev, rk, rv, prob.spec.name)
    # rows past each context's end stay untouched (NaN)
    gk = U.dev_to_f64(dev.tgt_k, prob.spec.dtype)
    for b, t in enumerate(prob.tgt_tokens):
        assert np.isnan(gk[:, b, :, int(t):]).all(), "row past the context's end was written"
    dev.close()


def test_batch_over_one_launch():
    """70 contexts: the host splits them into launches of 64 and 6."""
    _check(S.make_problem(_spec(name="batch70", src_tokens=24, batch=70)))


def test_single_source_token():
    _check(S.make_problem(_spec(name="one-token", src_tokens=1, batch=3)))


def test_empty_contexts_and_rows():
    """Hand-made alignment: a context with no target tokens, rows with no
    entries (bias-only output), entries out of order and repeated."""
    spec = _spec(name="empty-rows", src_tokens=37, batch=3, span_lo=1, span_hi=2)
    prob = S.make_problem(spec)
    rng = np.random.default_rng(5)
    tt = np.array([0, 5, 37], dtype=np.int32)
    counts = []
    cols = []
    for b, t in enumerate(tt):
        for r in range(int(t)):
            n = int(rng.integers(0, 4)) if r % 4 else 0   # every 4th row empty
            counts.append(n)
            cols.extend(int(x) for x in rng.integers(0, spec.src_tokens, size=n))
    row_ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    col_idx = np.array(cols, dtype=np.int32)
    weight = rng.uniform(-1.0, 1.0, size=len(cols)).astype(np.float32)
    prob = dataclasses.replace(prob, tgt_tokens=tt, row_ptr=row_ptr, col_idx=col_idx,
                               weight=weight)
    _check(prob)


def test_long_spans():
    """Rows pooling 3 to 7 source tokens (the fused kernel prefetches the
    second entry, requests the third entry's index early and reads the rest
    in its pooling loop), drawn spans and a hand-made map with entries out
    of order, repeated, and weights of both signs; split and fp16 operand
    precisions."""
    spec = _spec(name="long-spans", src_tokens=700, batch=2, span_lo=3, span_hi=7)
    prob = S.make_problem(spec)
    _check(prob)
    _check(prob, precision=kvx.KVX_PREC_F16)
    rng = np.random.default_rng(11)
    tt = np.array([90, 161], dtype=np.int32)
    counts, cols = [], []
    for t in tt:
        for r in range(int(t)):
            n = int(rng.integers(3, 8))
            counts.append(n)
            cols.extend(int(x) for x in rng.integers(0, spec.src_tokens, size=n))
    row_ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    weight = rng.uniform(-1.0, 1.0, size=len(cols)).astype(np.float32)
    _check(dataclasses.replace(prob, tgt_tokens=tt, row_ptr=row_ptr,
                               col_idx=np.array(cols, dtype=np.int32), weight=weight))


def test_two_heads_per_chunk_mix2_partial_tile():
    """Ds = 64 (a K-chunk spans two source heads), two mixed source layers,
    and dout = 384 (the second output tile is half used)."""
    spec = _spec(name="ds64-mix2-dout384", src=S.ModelShape(4, 2, 64, 1.0e4),
                 tgt=S.ModelShape(2, 3, 128, 1.0e6), mix=2, layer_map=(0, 1, 3, 2),
                 src_tokens=200, batch=2)
    _check(S.make_problem(spec))
    _check(S.make_problem(dataclasses.replace(spec, name="ds64-mix2-spans", span_lo=1,
                                              span_hi=2)))
    _check(S.make_problem(spec), precision=kvx.KVX_PREC_F16)


def test_interleaved_tile_order():
    """din = 1024 (two mixed source layers of 4 heads x 128) selects the
    interleaved tile order.  More work units than compute units, so each
    workgroup steps through several of them (carries across N tile, row
    tile, K|V and layer); dout = 384 leaves the second N tile half used.
    Identity alignment, span maps and the F16 operand mode."""
    spec = _spec(name="interleaved", src=S.ModelShape(4, 4, 128, 1.0e6),
                 tgt=S.ModelShape(4, 3, 128, 1.0e4), mix=2,
                 layer_map=(0, 1, 1, 2, 2, 3, 3, 0), src_tokens=1100, batch=3)
    prob = S.make_problem(spec)
    # more work units (row tiles x N tiles x layers x K|V) than compute units
    n_cu = U.torch().cuda.get_device_properties(0).multi_processor_count
    units = sum(-(-int(t) // 128) for t in prob.tgt_tokens) * 2 * 4 * 2
    assert units > n_cu, (units, n_cu)
    _check(prob, expect_order=1)
    _check(prob, precision=kvx.KVX_PREC_F16, expect_order=1)
    spans = S.make_problem(dataclasses.replace(spec, name="interleaved-spans", batch=4,
                                               span_lo=1, span_hi=3))
    _check(spans, expect_order=1)
    # a shorter contraction keeps the contiguous order
    short = S.make_problem(dataclasses.replace(spec, name="contiguous", mix=1,
                                               layer_map=(0, 1, 2, 3), src_tokens=300))
    _check(short, expect_order=0)


def test_resident_order_shapes():
    """The resident order (span maps, din <= 256, several N tiles): a single
    K-chunk (din 128) with a partly used second N tile, two chunks with
    three N tiles over more row-tile groups than compute units (so that
    workgroup ranges begin and end inside groups), and ragged contexts."""
    one = _spec(name="resident-1chunk", src=S.ModelShape(2, 1, 128, 1.0e6),
                tgt=S.ModelShape(2, 3, 128, 1.0e4), layer_map=(1, 0), src_tokens=700, batch=3,
                span_lo=1, span_hi=3)
    _check(S.make_problem(one), expect_order=2)
    _check(S.make_problem(one), precision=kvx.KVX_PREC_F16, expect_order=2)
    two = _spec(name="resident-groups", src=S.ModelShape(3, 2, 128, 1.0e6),
                tgt=S.ModelShape(2, 6, 128, 1.0e4), layer_map=(2, 0), src_tokens=2000,
                batch=9, span_lo=1, span_hi=2)
    prob = S.make_problem(two)
    n_cu = U.torch().cuda.get_device_properties(0).multi_processor_count
    groups = sum(-(-int(t) // 128) for t in prob.tgt_tokens) * 2 * 2
    assert groups > n_cu, (groups, n_cu)
    _check(prob, expect_order=2)
    # identity alignment on such a plan takes the contiguous order
    _check(S.make_problem(dataclasses.replace(two, name="resident-plan-identity", span_lo=0,
                                              span_hi=0, batch=2, src_tokens=300)))


def test_strided_source_view():
    """Source K/V are views into larger caches (extra tokens after T_s)."""
    T = U.torch()
    spec = _spec(name="strided", src_tokens=100, batch=2)
    prob = S.make_problem(spec)
    print(f"[edges] {spec.name}", flush=True)
    dev = U.DevProblem(prob)
    pad = 24
    Ls, B, Hs, Ts, Ds = prob.src_k.shape
    big_k = T.full((Ls, B, Hs, Ts + pad, Ds), float("nan"), dtype=T.bfloat16, device="cuda")
    big_v = T.full_like(big_k, float("nan"))
    big_k[:, :, :, :Ts] = dev.src_k
    big_v[:, :, :, :Ts] = dev.src_v
    strides = tuple(int(x) for x in big_k.stride()[:4])
    dev.tr(big_k[:, :, :, :Ts], big_v[:, :, :, :Ts], dev.tgt_k, dev.tgt_v, dev.cap,
           src_stride=strides)
    T.cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    U.check_full(dev, rk, rv, spec.name)
    dev.close()


def test_misaligned_layout_refused():
    """A bf16 plan runs the fused kernel, which needs 16-byte aligned rows: an
    odd token stride is refused with KVX_EUNSUPPORTED before any launch."""
    T = U.torch()
    prob = S.make_problem(_spec(name="misaligned", src_tokens=16))
    dev = U.DevProblem(prob)
    Ls, B, Hs, Ts, Ds = prob.src_k.shape
    odd = (B * Hs * Ts * (Ds + 1), Hs * Ts * (Ds + 1), Ts * (Ds + 1), Ds + 1)
    buf = T.zeros(Ls * odd[0], dtype=T.bfloat16, device="cuda")
    io, keep = kvx.make_io(B, Ts, buf, buf, dev.tgt_k, dev.tgt_v, dev.cap, src_stride=odd)
    st = kvx.kvx_translate_status(dev.tr.plan, io, T.cuda.current_stream().cuda_stream)
    assert st == kvx.KVX_EUNSUPPORTED
    dev.close()
