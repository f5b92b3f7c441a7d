"""Bit-exact GPU probes of the translation's integer work -- the layer map,
layer mixing, head and token addressing, the consumption of the alignment
CSR and both tile orders -- and of NaN locality.

Exactness.  With RoPE off on both sides (rope_base 0: every angle is 0, so
cos = 1 and sin = 0 exactly), source K/V small integers in [-4, 4], pooling
weights 1, 1/2 and 1/4 over rows of 1, 2 and 4 entries (pooled values are
multiples of 1/4 in [-4, 4]) and translator rows holding at most six nonzero
weights +-1 or +-2 (|u| <= 24), every intermediate of the operator is exactly
representable: the bf16 operand (the split's low part is zero), every fp32
partial sum, and the bf16 output (a multiple of 1/4 below 64 needs at most 8
significant bits).  The GPU output must then equal the fp64 oracle bit for
bit, in every precision mode.  The translator rows are drawn so that every
input feature of every target layer feeds some output, so a misrouted source
layer, head, token, feature or alignment entry changes some value.

Shapes: the Qwen2.5-7B -> 1.5B geometry (identity alignment, one N tile),
Qwen2.5-1.5B -> Gemma-2-2B (its round(27 l / 25) layer map, four N tiles,
spans, several contexts) and Llama3.1-70B -> Qwen2.5-7B (3-layer windows that
read layers 2, 22, 42 and 62 twice, the interleaved tile order), each over
several row tiles with a ragged last one.
"""
import dataclasses

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

MODES = [kvx.KVX_PREC_BF16X2, kvx.KVX_PREC_BF16, kvx.KVX_PREC_F16, kvx.KVX_PREC_BF16X2_OUTLIER]
MODE_ID = {kvx.KVX_PREC_BF16X2: "bf16x2", kvx.KVX_PREC_BF16: "bf16", kvx.KVX_PREC_F16: "f16",
           kvx.KVX_PREC_BF16X2_OUTLIER: "outlier"}
BF16_NAN = np.uint16(0x7FC0)


def _no_rope(spec):
    return spec.replace(src=dataclasses.replace(spec.src, rope_base=0.0),
                        tgt=dataclasses.replace(spec.tgt, rope_base=0.0), outliers=0)


def _pow2_lengths(rng, n_tokens):
    """Row lengths from {1, 2, 4} covering n_tokens; a remainder too short for
    the drawn length takes the largest power of two that fits."""
    lens, left = [], n_tokens
    while left > 0:
        n = int(rng.choice([1, 2, 4]))
        while n > left:
            n //= 2
        lens.append(n)
        left -= n
    return np.array(lens, dtype=np.int64)


def _pow2_csr(rng, batch, n_tokens, scattered):
    """Alignment rows of 1, 2 or 4 entries with weight 1/len each.  Spans
    (contiguous source tokens, in order) or, with ``scattered``, entries drawn
    anywhere in the context (repeats allowed) in random order."""
    counts, cols = [], []
    tt = []
    for _ in range(batch):
        lens = _pow2_lengths(rng, n_tokens)
        tt.append(len(lens))
        start = 0
        for n in lens:
            if scattered:
                c = rng.integers(0, n_tokens, size=n)
            else:
                c = rng.permutation(np.arange(start, start + n)) if n > 1 else [start]
            cols.extend(int(x) for x in c)
            counts.append(int(n))
            start += n
    row_ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    weight = np.repeat(1.0 / np.array(counts, dtype=np.float64), counts).astype(np.float32)
    return (np.array(tt, dtype=np.int32), row_ptr, np.array(cols, dtype=np.int32), weight)


def _selection_w(rng, lt, dout, din):
    """[lt, dout, din] with m = clip(ceil(din / dout), 2, 6) nonzero weights per
    row, +-1 or +-2 (only +-1 when m > 3); the columns come from concatenated
    permutations, so every input feature is used at least once."""
    m = min(6, max(2, -(-din // dout)))
    coef = np.array([1.0, -1.0, 2.0, -2.0] if m <= 3 else [1.0, -1.0], dtype=np.float32)
    w = np.zeros((lt, dout, din), dtype=np.float32)
    reps = -(-m * dout // din)
    for l in range(lt):
        cols = np.concatenate([rng.permutation(din) for _ in range(reps)])[:m * dout]
        cols = cols.reshape(dout, m)
        rows = np.repeat(np.arange(dout), m).reshape(dout, m)
        np.add.at(w[l], (rows, cols), rng.choice(coef, size=(dout, m)))
    return w


def _exact_problem(cfg, T, B, scattered=False, seed=0):
    spec = _no_rope(S.config(cfg, src_tokens=T, batch=B))
    rng = np.random.default_rng([seed, cfg, T, B, int(scattered)])
    prob = S.make_problem(spec)
    shape = prob.src_k.shape
    prob.src_k = S.to_storage(rng.integers(-4, 5, size=shape).astype(np.float32), S.BF16)
    prob.src_v = S.to_storage(rng.integers(-4, 5, size=shape).astype(np.float32), S.BF16)
    lt, dout, din = spec.tgt.n_layers, spec.d_out, spec.d_in
    prob.w_k = S.to_storage(_selection_w(rng, lt, dout, din), S.BF16)
    prob.w_v = S.to_storage(_selection_w(rng, lt, dout, din), S.BF16)
    if not spec.identity_align:
        tt, rp, ci, w = _pow2_csr(rng, B, T, scattered)
        prob = dataclasses.replace(prob, tgt_tokens=tt, row_ptr=rp, col_idx=ci, weight=w)
    return prob


def _marks(prob, rng):
    """Random outlier marks for KVX_PREC_BF16X2_OUTLIER (5% of the channels),
    so that split and unsplit k-steps both occur."""
    s = prob.spec.src
    shape = (s.n_layers, s.n_kv_heads, s.head_dim)
    return rng.random(shape) < 0.05, rng.random(shape) < 0.05


def _assert_bitwise(got, ref, what):
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    if not same.all():
        bad = np.argwhere(~same)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {got.size} elements differ; first at "
                             f"{i}: gpu {got[i]!r} oracle {ref[i]!r}")


def _run_exact(prob, precision, expect_order=None):
    spec = prob.spec
    print(f"[probe] {spec.name} T={spec.src_tokens} B={spec.batch} {MODE_ID[precision]} "
          f"tt={list(prob.tgt_tokens)}", flush=True)
    outl = _marks(prob, np.random.default_rng(1)) \
        if precision == kvx.KVX_PREC_BF16X2_OUTLIER else None
    dev = U.DevProblem(prob, precision, outliers=outl)
    info = dev.tr.info()
    assert info.kernel == 1
    if expect_order is not None:
        assert info.tile_order == expect_order
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    for r in (rk, rv):  # the exact result is a bf16 value (the probe's premise)
        x = r[~np.isnan(r)].astype(np.float32)
        assert np.array_equal(S.bf16_bits_to_f32(S.f32_to_bf16_bits(x)), x)
    gk = U.dev_to_f64(dev.tgt_k, spec.dtype)
    gv = U.dev_to_f64(dev.tgt_v, spec.dtype)
    # rows past a context's end: NaN on both sides (untouched / not computed)
    _assert_bitwise(gk, rk, f"{spec.name} K")
    _assert_bitwise(gv, rv, f"{spec.name} V")
    # the probe is not vacuous: outputs reach well beyond one input's range,
    # and pooled rows produce fractions
    valid = ~np.isnan(rk)
    assert np.abs(rk[valid]).max() >= 8
    if not spec.identity_align:
        assert (rk[valid] != np.round(rk[valid])).any()
    dev.close()


@pytest.mark.parametrize("precision", MODES, ids=MODE_ID.get)
def test_exact_qwen7b_identity(precision):
    """1:1 layer map, identity alignment, 300 tokens (3 row tiles, ragged)."""
    _run_exact(_exact_problem(2, 300, 1), precision, expect_order=0)


@pytest.mark.parametrize("precision", MODES, ids=MODE_ID.get)
def test_exact_gemma_map_spans(precision):
    """round(27 l / 25) map (skips source layers 7 and 20), four N tiles,
    power-of-two spans, 3 contexts of different lengths."""
    _run_exact(_exact_problem(3, 700, 3), precision, expect_order=2)


@pytest.mark.parametrize("precision", MODES, ids=MODE_ID.get)
def test_exact_llama_windows_spans(precision):
    """3-layer windows (din 3072, interleaved tile order), spans of 1-4,
    2 contexts of 4 row tiles each."""
    _run_exact(_exact_problem(5, 700, 2), precision, expect_order=1)


@pytest.mark.parametrize("cfg", [3, 5])
def test_exact_scattered_entries(cfg):
    """Rows gathering 1, 2 or 4 tokens from anywhere in the context, in random
    order and with repeats."""
    _run_exact(_exact_problem(cfg, 400, 2, scattered=True), kvx.KVX_PREC_BF16X2)


def test_exact_batched_contexts():
    """8 contexts per call (the batched sweep's launch shape) at 520 tokens."""
    _run_exact(_exact_problem(4, 520, 8), kvx.KVX_PREC_BF16X2)


@pytest.mark.parametrize("precision", [kvx.KVX_PREC_BF16X2, kvx.KVX_PREC_F16], ids=MODE_ID.get)
def test_identity_csr_equals_identity_alignment(precision):
    """A CSR with one entry of weight 1 per row (row t reads token t) takes the
    span-map path of the kernel; on real data (RoPE on, outlier channels) it
    must give the same bits as identity alignment."""
    spec = S.config(2, src_tokens=300, batch=2)
    prob = S.make_problem(spec)
    T, B = spec.src_tokens, spec.batch
    print(f"[probe] identity CSR vs NULL alignment {MODE_ID[precision]}", flush=True)
    a = U.DevProblem(prob, precision)
    a.run()
    csr = dataclasses.replace(prob, tgt_tokens=np.full(B, T, dtype=np.int32),
                              row_ptr=np.arange(B * T + 1, dtype=np.int32),
                              col_idx=np.tile(np.arange(T, dtype=np.int32), B),
                              weight=np.ones(B * T, dtype=np.float32))
    b = U.DevProblem(csr, precision)
    b.run()
    U.torch().cuda.synchronize()
    for x, y, name in ((a.tgt_k, b.tgt_k, "K"), (a.tgt_v, b.tgt_v, "V")):
        gx, gy = U.dev_to_f64(x, spec.dtype), U.dev_to_f64(y, spec.dtype)
        assert np.isfinite(gx).all()
        _assert_bitwise(gy, gx, f"identity CSR {name}")
    a.close()
    b.close()


def _readers(spec, ls):
    """Target layers whose window reads source layer ls."""
    m = spec.mix
    return sorted({l for l in range(spec.tgt.n_layers)
                   for j in range(m) if spec.layer_map[l * m + j] == ls})


@pytest.mark.parametrize("cfg,T,ls,skipped", [(3, 500, 5, 7), (5, 300, 2, None)])
def test_nan_locality(cfg, T, ls, skipped):
    """A NaN in one element of source K (layer ls, context 1, head 1, token k,
    channel 5) reaches exactly the target rows of context 1 whose alignment
    row reads token k, in exactly the target layers whose window reads ls, in
    every feature of K and nowhere in V.  A NaN in a source layer no window
    reads (Gemma's map skips layer 7) reaches nothing."""
    spec = S.config(cfg, src_tokens=T, batch=2)
    prob = S.make_problem(spec)
    k = T // 2 + 3
    prob.src_k[ls, 1, 1, k, 5] = BF16_NAN
    if skipped is not None:
        assert _readers(spec, skipped) == []
        prob.src_k[skipped, 0, 0, 10, 0] = BF16_NAN
    readers = _readers(spec, ls)
    assert readers and (cfg != 5 or len(readers) == 2)
    print(f"[probe] NaN locality {spec.name}: source layer {ls} read by {readers}", flush=True)
    dev = U.DevProblem(prob)
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    gk = U.dev_to_f64(dev.tgt_k, spec.dtype)
    gv = U.dev_to_f64(dev.tgt_v, spec.dtype)
    tt = prob.tgt_tokens
    off = prob.row_offsets()
    rows1 = [t for t in range(int(tt[1]))
             if k in set(prob.col_idx[prob.row_ptr[off[1] + t]:prob.row_ptr[off[1] + t + 1]])]
    assert rows1
    expect = np.zeros(gk.shape, dtype=bool)
    for l in readers:
        for t in rows1:
            expect[l, 1, :, t, :] = True
    for b in range(spec.batch):
        v = slice(0, int(tt[b]))
        assert np.array_equal(np.isnan(gk[:, b, :, v]), expect[:, b, :, v]), \
            f"context {b}: NaN pattern of K differs from the expected rows"
        assert np.array_equal(np.isnan(rk[:, b, :, v]), expect[:, b, :, v])
        assert not np.isnan(gv[:, b, :, v]).any(), "NaN reached V"
        fin = ~expect[:, b, :, v]
        U.check_close(gk[:, b, :, v][fin], rk[:, b, :, v][fin], spec.dtype, "finite K")
        U.check_close(gv[:, b, :, v].reshape(-1), rv[:, b, :, v].reshape(-1), spec.dtype,
                      "V")
    dev.close()
