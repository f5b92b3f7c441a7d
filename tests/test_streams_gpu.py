"""Serving-style use of kvx_translate on the GPU: capture into a HIP graph
and replay, and concurrent calls on two streams.

* The call path enqueues kernels only (no allocation, copy, memset or
  synchronisation unless KVX_VALIDATE=1), so a translation captured into a
  graph replays to the eager result bit for bit -- checked on several
  replays, with eager work and synchronisations between them, and with the
  targets refilled before each replay so a replay that did nothing fails.
* A plan holds no per-call scratch, so calls of two plans on two streams
  (default priority) may overlap; each stream's result equals its eager
  single-stream result bit for bit.
"""
import dataclasses
import os

import numpy as np
import pytest

from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

QWEN_SMALL = S.ModelShape(2, 4, 128, 1.0e6)


def _spec(**kw):
    base = dict(cfg_id=600, name="streams", src=QWEN_SMALL, tgt=S.ModelShape(2, 2, 128, 1.0e6),
                mix=1, layer_map=(1, 0), dtype=S.BF16, src_tokens=300, batch=2, outliers=4,
                bias_std=0.5, seed=9)
    base.update(kw)
    return S.Spec(**base)


def _bits(t):
    T = U.torch()
    return t.view(T.int16).clone()


@pytest.mark.parametrize("spans", [False, True])
def test_graph_capture_replays(spans):
    assert os.environ.get("KVX_VALIDATE", "0") != "1"
    T = U.torch()
    spec = _spec(name=f"graph-{spans}", **({"span_lo": 1, "span_hi": 3} if spans else {}))
    prob = S.make_problem(spec)
    print(f"[streams] {spec.name}", flush=True)
    dev = U.DevProblem(prob, cap=max(1, int(prob.tgt_tokens.max())))
    dev.run()
    T.cuda.synchronize()
    ref_k, ref_v = _bits(dev.tgt_k), _bits(dev.tgt_v)
    g = T.cuda.CUDAGraph()
    side = T.cuda.Stream()
    side.wait_stream(T.cuda.current_stream())
    with T.cuda.stream(side):
        with T.cuda.graph(g, stream=side):
            dev.run()  # the current stream is the capturing one
    T.cuda.synchronize()
    prob2 = S.make_problem(dataclasses.replace(spec, seed=10))
    other = U.DevProblem(prob2, cap=max(1, int(prob2.tgt_tokens.max())))
    for rep in range(3):
        dev.tgt_k.fill_(float("nan"))
        dev.tgt_v.fill_(float("nan"))
        T.cuda.synchronize()
        g.replay()
        other.run()  # eager work of another plan between replays
        T.cuda.synchronize()
        assert T.equal(_bits(dev.tgt_k), ref_k), f"replay {rep}: K differs"
        assert T.equal(_bits(dev.tgt_v), ref_v), f"replay {rep}: V differs"
    other.close()
    dev.close()


def test_two_streams_concurrent():
    T = U.torch()
    a = U.DevProblem(S.make_problem(_spec(name="stream-a", span_lo=1, span_hi=3)))
    b = U.DevProblem(S.make_problem(_spec(name="stream-b", seed=11, src_tokens=520)))
    print("[streams] eager references", flush=True)
    a.run()
    b.run()
    T.cuda.synchronize()
    refs = [(_bits(a.tgt_k), _bits(a.tgt_v)), (_bits(b.tgt_k), _bits(b.tgt_v))]
    s1, s2 = T.cuda.Stream(), T.cuda.Stream()
    for d in (a, b):
        d.tgt_k.fill_(float("nan"))
        d.tgt_v.fill_(float("nan"))
    T.cuda.synchronize()
    print("[streams] overlapped calls", flush=True)
    for _ in range(4):
        a.run(stream=s1)
        b.run(stream=s2)
    T.cuda.synchronize()
    for d, (rk, rv), name in ((a, refs[0], "a"), (b, refs[1], "b")):
        assert T.equal(_bits(d.tgt_k), rk), f"stream {name}: K differs"
        assert T.equal(_bits(d.tgt_v), rv), f"stream {name}: V differs"
    a.close()
    b.close()
