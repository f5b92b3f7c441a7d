"""Failure handling forced from the host: with KVX_FAULT=launch a call that
passes validation reports a failed launch (KVX_EHIP, hipErrorLaunchFailure)
and enqueues nothing, so the target cache keeps its previous contents; the
next call without the variable runs normally.  This is the path a runtime
takes to its fallback (native prefill) when a translation is unavailable.
No kernel is made to fail: the library returns before any launch.
"""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

HIP_ERROR_LAUNCH_FAILURE = 719


@pytest.fixture
def fault_env():
    old = os.environ.get("KVX_FAULT")
    yield
    if old is None:
        os.environ.pop("KVX_FAULT", None)
    else:
        os.environ["KVX_FAULT"] = old


def _io(dev):
    prob, spec = dev.prob, dev.spec
    ident = prob.row_ptr is None
    return kvx.make_io(spec.batch, spec.src_tokens, dev.src_k, dev.src_v, dev.tgt_k, dev.tgt_v,
                       dev.cap, None if ident else prob.tgt_tokens, dev.row_ptr, dev.col_idx,
                       dev.weight)


def _untouched(dev):
    T = U.torch()
    T.cuda.synchronize()
    return bool(T.isnan(dev.tgt_k).all()) and bool(T.isnan(dev.tgt_v).all())


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_injected_launch_fault_then_recovery(cfg, fault_env):
    spec = S.config(cfg, src_tokens=260, batch=2)
    prob = S.make_problem(spec)
    print(f"[fault] {spec.name} KVX_FAULT=launch", flush=True)
    dev = U.DevProblem(prob)
    io, keep = _io(dev)
    os.environ["KVX_FAULT"] = "launch"
    st = kvx.kvx_translate_status(dev.tr.plan, io, U.torch().cuda.current_stream().cuda_stream)
    assert st == kvx.KVX_EHIP, kvx.status_string(st)
    assert kvx.load().kvx_last_hip_error() == HIP_ERROR_LAUNCH_FAILURE
    assert _untouched(dev), "a failed call wrote the target cache"
    # validation still comes first: a bad descriptor is reported as such
    bad, bkeep = kvx.make_io(spec.batch, spec.src_tokens, dev.src_k, dev.src_v, dev.tgt_k,
                             dev.tgt_v, 0, None if prob.row_ptr is None else prob.tgt_tokens,
                             dev.row_ptr, dev.col_idx, dev.weight)
    assert kvx.kvx_translate_status(dev.tr.plan, bad) != kvx.KVX_EHIP
    del bkeep
    # recovery: the same plan and buffers, without the fault
    del os.environ["KVX_FAULT"]
    print(f"[fault] {spec.name} recovery", flush=True)
    dev.run()
    U.torch().cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    U.check_full(dev, rk, rv, f"after fault {spec.name}", 0.75)
    del keep
    dev.close()


def test_injected_launch_fault_staged(fault_env):
    T = U.torch()
    spec = S.config(2, src_tokens=260)
    prob = S.make_problem(spec)
    print("[fault] staged KVX_FAULT=launch", flush=True)
    dev = U.DevProblem(prob)
    io, keep = _io(dev)
    n = kvx.kvx_staged_workspace_bytes(dev.tr.plan, io, spec.tgt.n_layers)
    ws = T.empty(n, dtype=T.uint8, device="cuda")
    os.environ["KVX_FAULT"] = "launch"
    st = kvx.kvx_translate_staged_status(dev.tr.plan, io, ws.data_ptr(), n)
    assert st == kvx.KVX_EHIP, kvx.status_string(st)
    assert _untouched(dev)
    del os.environ["KVX_FAULT"]
    kvx.kvx_translate_staged(dev.tr.plan, io, ws)
    T.cuda.synchronize()
    rk, rv = O.translate(prob, cap=dev.cap)
    U.check_full(dev, rk, rv, "staged after fault", 0.75)
    del keep
    dev.close()
