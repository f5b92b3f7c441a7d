"""The seeded input generator: layer maps, span maps, casts, determinism."""
import os

import numpy as np
import pytest

from paper_2608_30963_amd import synth as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "layer_maps.txt")


def _golden():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, *vals = line.split()
        out[name] = [int(v) for v in vals]
    return out


def test_layer_maps_match_rational_enumeration():
    g = _golden()
    assert list(S.config(3).layer_map) == g["qwen1.5b_to_gemma2b"]
    assert list(S.config(4).layer_map) == g["qwen1.5b_to_gemma2b"]
    m5 = S.config(5).layer_map
    starts = g["llama70b_to_qwen7b_window_start"]
    assert list(m5) == [s + j for s in starts for j in range(3)]
    # every source layer of the 80 is read, layers 7 and 20 of Qwen are skipped
    assert set(m5) == set(range(80))
    assert {7, 20}.isdisjoint(S.config(3).layer_map)
    assert list(S.config(2).layer_map) == list(range(28))


@pytest.mark.parametrize("cfg,lo,hi", [(3, 1, 3), (5, 1, 2)])
def test_spans_partition_source(cfg, lo, hi):
    spec = S.config(cfg, src_tokens=997, batch=3)
    tt, rp, ci, w = S.span_csr(spec)
    assert rp[0] == 0 and np.all(np.diff(rp) >= 1)
    assert len(rp) == tt.sum() + 1
    off = 0
    for b in range(spec.batch):
        rows = rp[off:off + tt[b] + 1]
        cols = ci[rows[0]:rows[-1]]
        # each source token appears exactly once, in order
        assert np.array_equal(cols, np.arange(spec.src_tokens))
        lens = np.diff(rows)
        assert lens[:-1].min() >= lo and lens.max() <= hi
        for r in range(tt[b]):
            ws = w[rows[r]:rows[r + 1]]
            assert np.all(ws == np.float32(1.0 / len(ws)))
            assert abs(float(ws.astype(np.float64).sum()) - 1.0) <= len(ws) * 2.0 ** -23
        off += tt[b]


def test_span_count_near_expectation():
    spec = S.config(3)
    tt, *_ = S.span_csr(spec)
    assert abs(int(tt[0]) - 4096 / 2) < 100


def test_bf16_cast_is_rne():
    import torch
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 30
    x[:4] = [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 65504.0]
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(S.f32_to_bf16_bits(x), want)
    assert np.array_equal(S.bf16_bits_to_f32(want), torch.from_numpy(want.view(np.int16))
                          .view(torch.bfloat16).float().numpy())


def test_outliers_and_determinism():
    spec = S.config(2, src_tokens=64).replace(src=S.ModelShape(2, 4, 128, 1e6),
                                               tgt=S.ModelShape(2, 2, 128, 1e6),
                                               layer_map=(0, 1))
    a = S.draw_source(spec, 0)
    b = S.draw_source(spec, 0)
    assert np.array_equal(a, b)
    big = np.abs(a).max(axis=3) > 8          # [L, B, H, D] channels with outliers
    assert np.all(big.sum(axis=-1) == 4)
    # a subset draw gives identical layers
    c = S.draw_source(spec, 0, layers=[1])
    assert np.array_equal(c[1], a[1]) and not c[0].any()


def test_weight_scale():
    spec = S.config(3)
    w = S.draw_weights(spec.replace(tgt=S.ModelShape(2, 4, 256, 1e4), layer_map=(0, 1)), 0)
    assert abs(w.std() * np.sqrt(256) - 1.0) < 0.01
