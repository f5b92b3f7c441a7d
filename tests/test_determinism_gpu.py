"""Run-to-run determinism: the same translation, run twice into fresh
buffers, gives the same bits.  The kernels pool, contract and reduce in a
fixed order with no atomics, so any difference would come from a race on
the LDS buffers the producer and consumer waves share (or a read of
uninitialised memory) -- the race detector of this library.  Covers the
identity, span-map and layer-window workloads in every precision mode, eight
contexts per call, a paged target and the staged path.
"""
import numpy as np
import pytest

from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

PRECS = [kvx.KVX_PREC_BF16X2, kvx.KVX_PREC_BF16, kvx.KVX_PREC_F16]


def _twice(prob, precision, fill_b=-7.0):
    """Outputs of two runs; the second into buffers pre-filled differently,
    so a row written by only one of the runs shows up too."""
    spec = prob.spec
    a = U.DevProblem(prob, precision)
    a.run()
    b = U.DevProblem(prob, precision, fill=fill_b)
    b.run()
    U.torch().cuda.synchronize()
    out = []
    tt = prob.tgt_tokens
    for x, y in ((a.tgt_k, b.tgt_k), (a.tgt_v, b.tgt_v)):
        gx, gy = U.dev_to_f64(x, spec.dtype), U.dev_to_f64(y, spec.dtype)
        for bb in range(spec.batch):
            out.append((gx[:, bb, :, :tt[bb]], gy[:, bb, :, :tt[bb]]))
    a.close()
    b.close()
    return out


@pytest.mark.parametrize("cfg,T,B", [(2, 700, 1), (3, 900, 2), (4, 300, 8), (5, 520, 1)])
@pytest.mark.parametrize("precision", PRECS, ids=["bf16x2", "bf16", "f16"])
def test_same_bits_twice(cfg, T, B, precision):
    spec = S.config(cfg, src_tokens=T, batch=B)
    print(f"[determinism] {spec.name} T={T} B={B} prec {precision}", flush=True)
    for x, y in _twice(S.make_problem(spec), precision):
        assert np.isfinite(x).all() and np.isfinite(y).all()
        assert np.array_equal(x, y), f"{spec.name}: runs differ in {int((x != y).sum())} elements"


def test_same_bits_twice_paged():
    T = U.torch()
    spec = S.config(3, src_tokens=700, batch=2)
    prob = S.make_problem(spec)
    print("[determinism] paged", flush=True)
    bs = 16
    need = [(int(t) + bs - 1) // bs for t in prob.tgt_tokens]
    perm = np.random.default_rng(3).permutation(sum(need)).astype(np.int32)
    table = np.zeros((spec.batch, max(need)), dtype=np.int32)
    k = 0
    for bb, n in enumerate(need):
        table[bb, :n] = perm[k:k + n]
        k += n
    bt = T.from_numpy(table).cuda()
    shape = (spec.tgt.n_layers, int(perm.size), spec.tgt.n_kv_heads, bs, spec.tgt.head_dim)
    dev = U.DevProblem(prob)
    outs = []
    for fill in (float("nan"), -7.0):
        tk = T.full(shape, fill, dtype=T.bfloat16, device="cuda")
        tv = T.full(shape, fill, dtype=T.bfloat16, device="cuda")
        dev.tr(dev.src_k, dev.src_v, tk, tv, None, prob.tgt_tokens, dev.row_ptr, dev.col_idx,
               dev.weight, block_table=bt, block_size=bs)
        T.cuda.synchronize()
        outs.append((tk.float().cpu().numpy(), tv.float().cpu().numpy()))
    # every block the table uses holds the same bits; unused slots keep each fill
    for bb, t in enumerate(prob.tgt_tokens):
        for j in range(int(t)):
            blk, slot = table[bb, j // bs], j % bs
            for h in range(2):
                assert np.array_equal(outs[0][h][:, blk, :, slot], outs[1][h][:, blk, :, slot])
    dev.close()


def test_same_bits_twice_staged():
    T = U.torch()
    spec = S.config(5, src_tokens=400)
    prob = S.make_problem(spec)
    print("[determinism] staged", flush=True)
    res = []
    for fill in (None, -7.0):
        dev = U.DevProblem(prob, fill=fill)
        io, keep = kvx.make_io(spec.batch, spec.src_tokens, dev.src_k, dev.src_v, dev.tgt_k,
                               dev.tgt_v, dev.cap, prob.tgt_tokens, dev.row_ptr, dev.col_idx,
                               dev.weight)
        n = kvx.kvx_staged_workspace_bytes(dev.tr.plan, io, spec.tgt.n_layers)
        ws = T.full((n,), 0x5a, dtype=T.uint8, device="cuda")
        kvx.kvx_translate_staged(dev.tr.plan, io, ws)
        T.cuda.synchronize()
        tt = int(prob.tgt_tokens[0])
        res.append((U.dev_to_f64(dev.tgt_k, spec.dtype)[:, :, :, :tt],
                    U.dev_to_f64(dev.tgt_v, spec.dtype)[:, :, :, :tt]))
        del keep
        dev.close()
    for h in range(2):
        assert np.array_equal(res[0][h], res[1][h])
