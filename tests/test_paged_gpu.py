"""GPU parity of the paged target layout (cache assembly through a block
table) against the fp64 oracle's contiguous result.

Every target row is read back from the physical block and slot its block
table entry names and compared with the oracle; every slot no target token
maps to must still hold the NaN the test filled it with (no stray writes).
"""
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_30963_amd import kvx, synth as S
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _block_table(tt, block_size, seed, spare=5):
    """Random distinct physical blocks for each context's logical blocks;
    unused entries hold -1 (never read)."""
    need = [(int(t) + block_size - 1) // block_size for t in tt]
    max_blocks = max(need) + 1
    num_blocks = sum(need) + spare
    perm = np.random.default_rng(seed).permutation(num_blocks).astype(np.int32)
    table = np.full((len(tt), max_blocks), -1, dtype=np.int32)
    k = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[k:k + n]
        k += n
    return table, num_blocks


def _run_paged(spec, block_size, precision=kvx.KVX_PREC_BF16X2, flash=False, seed=7,
               expect_order=None):
    T = U.torch()
    prob = S.make_problem(spec)
    tt = prob.tgt_tokens
    print(f"[paged] {spec.name} T={spec.src_tokens} B={spec.batch} bs={block_size} "
          f"flash={flash}", flush=True)
    table, nblk = _block_table(tt, block_size, seed)
    dev = U.DevProblem(prob, precision, cap=1)
    if expect_order is not None:
        assert dev.tr.info().tile_order == expect_order
    Lt, Ht, Dt = spec.tgt.n_layers, spec.tgt.n_kv_heads, spec.tgt.head_dim
    tdt = T.bfloat16 if spec.dtype == S.BF16 else T.float32
    if flash:  # [Lt][num_blocks][block_size][Ht][Dt]
        shape = (Lt, nblk, block_size, Ht, Dt)
        strides = (nblk * block_size * Ht * Dt, block_size * Ht * Dt, Dt, Ht * Dt)
    else:      # [Lt][num_blocks][Ht][block_size][Dt] (the default strides)
        shape = (Lt, nblk, Ht, block_size, Dt)
        strides = (0, 0, 0, 0)
    pk = T.full(shape, float("nan"), dtype=tdt, device="cuda")
    pv = T.full(shape, float("nan"), dtype=tdt, device="cuda")
    bt = T.from_numpy(table).cuda()
    ident = prob.row_ptr is None
    dev.tr(dev.src_k, dev.src_v, pk, pv, None, None if ident else tt, dev.row_ptr, dev.col_idx,
           dev.weight, tgt_stride=strides, block_table=bt, block_size=block_size)
    T.cuda.synchronize()
    rk, rv = O.translate(prob)
    gk, gv = U.dev_to_f64(pk, spec.dtype), U.dev_to_f64(pv, spec.dtype)
    if flash:  # to [Lt][num_blocks][Ht][block_size][Dt]
        gk, gv = gk.transpose(0, 1, 3, 2, 4), gv.transpose(0, 1, 3, 2, 4)
    written = np.zeros((nblk, block_size), dtype=bool)
    for b in range(spec.batch):
        t = np.arange(int(tt[b]))
        blk, slot = table[b, t // block_size], t % block_size
        written[blk, slot] = True
        for l in range(Lt):
            for name, g, r in (("K", gk, rk), ("V", gv, rv)):
                got = g[l, blk, :, slot, :]          # [tokens][Ht][Dt]
                ref = r[l, b].transpose(1, 0, 2)[:int(tt[b])]
                U.check_close(got.reshape(-1), ref.reshape(-1), spec.dtype,
                              f"paged {spec.name} ctx {b} layer {l} {name}")
    for g in (gk, gv):
        untouched = g.transpose(1, 3, 0, 2, 4)[~written]
        assert np.isnan(untouched).all(), "paged store touched a slot no token maps to"
    dev.close()


def test_paged_config2_identity():
    _run_paged(S.config(2, src_tokens=300), block_size=16)


def test_paged_config2_flash_layout_f16():
    _run_paged(S.config(2, src_tokens=257), block_size=32, precision=kvx.KVX_PREC_F16,
               flash=True)


def test_paged_config3_span_map_batch():
    """Span map with several N tiles: the resident order, rows stored through
    the block table from the consumers; also the flash-style layout."""
    _run_paged(S.config(3, src_tokens=700, batch=2), block_size=32, expect_order=2)
    _run_paged(S.config(3, src_tokens=500, batch=3), block_size=16, flash=True, expect_order=2)


def test_paged_config5_interleaved_span_map():
    """Long contraction (3 x 1024 features): interleaved tile order, span map,
    paged target."""
    _run_paged(S.config(5, src_tokens=300), block_size=16, expect_order=1)


def test_paged_config1_fp32_tiled():
    _run_paged(S.config(1, src_tokens=100, batch=3), block_size=8)


def _status(prob, dev, table, block_size, num_blocks, max_blocks=None):
    T = U.torch()
    Lt, Ht, Dt = prob.spec.tgt.n_layers, prob.spec.tgt.n_kv_heads, prob.spec.tgt.head_dim
    pk = T.zeros((Lt, num_blocks, Ht, max(block_size, 1), Dt), dtype=T.bfloat16, device="cuda")
    pv = T.zeros_like(pk)
    bt = T.from_numpy(table).cuda()
    io, keep = kvx.make_io(prob.spec.batch, prob.spec.src_tokens, dev.src_k, dev.src_v, pk, pv,
                           0, block_table=bt, block_size=block_size,
                           max_blocks=table.shape[1] if max_blocks is None else max_blocks,
                           num_blocks=num_blocks)
    st = kvx.kvx_translate_status(dev.tr.plan, io, T.cuda.current_stream().cuda_stream)
    T.cuda.synchronize()
    return st


def test_paged_argument_errors():
    prob = S.make_problem(S.config(2, src_tokens=64))
    dev = U.DevProblem(prob, cap=1)
    table, nblk = _block_table(prob.tgt_tokens, 16, seed=1)
    assert _status(prob, dev, table, 0, nblk) == kvx.KVX_EINVAL          # block_size 0
    assert _status(prob, dev, table, 16, 0) == kvx.KVX_EINVAL            # no blocks
    # 64 tokens need 4 blocks of 16: a table of 3 entries per context is short
    assert _status(prob, dev, table[:, :3].copy(), 16, nblk) == kvx.KVX_ESHAPE
    dev.close()


def test_paged_validation_mode_rejects_bad_block(monkeypatch):
    prob = S.make_problem(S.config(2, src_tokens=64))
    dev = U.DevProblem(prob, cap=1)
    table, nblk = _block_table(prob.tgt_tokens, 16, seed=2)
    table[0, 1] = nblk  # out of range
    monkeypatch.setenv("KVX_VALIDATE", "1")
    assert _status(prob, dev, table, 16, nblk) == kvx.KVX_EDATA
    table[0, 1] = 0
    monkeypatch.delenv("KVX_VALIDATE")
    dev.close()
