#!/usr/bin/env python3
"""Benchmark of the KV-translation operator on one MI355X.

A step is one ``kvx_translate`` call: every target layer's K and V of one
context, i.e. all stages of the translation (source-RoPE removal, alignment,
projection, target RoPE, store into the target cache layout).  Plan creation
(weight packing) happens once, before timing, as in serving.

Default workload: Qwen2.5-7B -> Qwen2.5-1.5B shaped KV caches at a 4K-token
context, bf16, same tokenizer (28 -> 28 layers, 4x128 -> 2x128 KV heads, RoPE
base 1e6 on both sides, 4 outlier channels per head scaled x20), seeded
synthetic data.  Inputs are resident in HBM before the timed region; three
buffer sets rotate so no call finds its inputs in the 256 MB last-level cache.

Prints one JSON line (rank 0).

``--fit`` measures the translator fit instead (include/kvx_fit.h): a step is
one ``kvx_fit_accumulate`` of the workload's paired caches (source cache and
a seeded stand-in for the target model's own cache) into every layer's K and
V normal equations; the solve is timed once afterwards.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFS = 2500.0    # MI355X dense bf16 matrix peak, TFLOP/s
METRIC = "translated tokens/s (all layers K+V) at 4K ctx; ms/handoff; % MFMA/HBM peak"


def algorithmic(spec, prob):
    """Bytes and flops the operator itself must move / compute per call:
    each used source element read once, each target element written once,
    translator weights read once, alignment map read once; flops of the
    pooled-then-projected contraction."""
    esz = 4 if spec.dtype == "f32" else 2
    used = len(set(int(x) for x in spec.layer_map))
    s = spec.src
    rows = int(prob.tgt_tokens.sum())
    read = 2 * used * spec.batch * s.n_kv_heads * spec.src_tokens * s.head_dim * esz
    write = 2 * spec.tgt.n_layers * rows * spec.d_out * esz
    weights = 2 * spec.tgt.n_layers * spec.d_out * spec.d_in * esz
    amap = 0 if prob.row_ptr is None else prob.row_ptr.nbytes + prob.col_idx.nbytes + \
        prob.weight.nbytes
    flops = 2 * 2 * spec.tgt.n_layers * rows * spec.d_in * spec.d_out
    return {"read": read, "write": write, "weights": weights, "map": amap,
            "bytes": read + write + weights + amap, "flops": flops}


KERNEL_SOURCES = os.path.join(ROOT, "paper_2608_30963_amd", "csrc")


def kernel_source_hash() -> str:
    """sha256 over the fused translation's HIP sources (file names and
    contents, sorted; the translator fit, the plan-time composition of
    translator variants and the staged path's separate kernels are not part
    of the fused launch)."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(KERNEL_SOURCES, "*"))):
        if os.path.basename(f) in ("fit.hip", "compose.hip", "staged.hip", "staged.h"):
            continue
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


PROFILES = os.path.join(ROOT, "profiles")


def recorded(workload: str, precision: str, src_tokens: int, batch: int, layout: str,
             key: str, profiles: str = None):
    """A value recorded in the committed rocprofv3 counter summary of this
    workload (profiles/*.md, "- key: value" lines), or None when no summary
    matches or the kernel sources have changed since the counters were
    taken: traffic_bytes_per_launch (FETCH_SIZE + WRITE_SIZE, scaled by a
    copy kernel's reading), mfma_busy_frac (SQ_VALU_MFMA_BUSY_CYCLES per SIMD
    over SQ_BUSY_CYCLES per shader engine)."""
    want = {"workload": workload, "precision": precision, "src_tokens": str(src_tokens),
            "batch": str(batch), "target_layout": layout,
            "kernel_source_sha256": kernel_source_hash()}
    for path in sorted(glob.glob(os.path.join(profiles or PROFILES, "*.md"))):
        rec = {}
        with open(path) as fh:
            for line in fh:
                if line.startswith("- ") and ": " in line:
                    k, v = line[2:].strip().split(": ", 1)
                    rec[k.strip("`")] = v.strip().strip("`")
        if all(rec.get(k) == v for k, v in want.items()) and key in rec:
            return rec[key]
    return None


def recorded_traffic(workload: str, precision: str, src_tokens: int, batch: int, layout: str,
                     profiles: str = None):
    """HBM bytes per launch (see recorded), or None."""
    v = recorded(workload, precision, src_tokens, batch, layout, "traffic_bytes_per_launch",
                 profiles)
    return None if v is None else int(v)


def gpu_clock_mhz():
    """The shader clock the driver reports as current (sysfs `pp_dpm_sclk`,
    the level marked `*`), sampled once while the timed calls run; None where
    the file is not readable.  A sample, not an average over the run."""
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            with open(path) as fh:
                for line in fh:
                    if line.strip().endswith("*"):
                        return int(line.split(":")[1].strip().split("Mhz")[0].split("MHz")[0])
        except (OSError, ValueError, IndexError):
            continue
    return None


def cpu_baseline(spec, prob, budget_s: float):
    """Time the fp64 oracle on the host: all target layers of a bounded
    number of tokens, scaled to source tokens per second."""
    from oracle import oracle as O
    lt = spec.tgt.n_layers
    n_tok = 16
    elapsed = 0.0
    while True:
        toks = np.linspace(0, int(prob.tgt_tokens[0]) - 1, n_tok).astype(np.int32)
        L = np.repeat(np.arange(lt, dtype=np.int32), n_tok)
        T = np.tile(toks, lt)
        B = np.zeros_like(L)
        t0 = time.perf_counter()
        O.rows(prob, L, B, T)
        elapsed = time.perf_counter() - t0
        if elapsed >= budget_s or n_tok >= int(prob.tgt_tokens[0]):
            break
        n_tok = min(int(prob.tgt_tokens[0]), max(n_tok * 2, int(n_tok * budget_s / max(elapsed, 1e-3) * 1.1)))
    # the whole context fits in less than the budget: repeat it
    passes = 1
    if elapsed < budget_s:
        passes = max(1, int(np.ceil(budget_s / max(elapsed, 1e-3))))
        t0 = time.perf_counter()
        for _ in range(passes):
            O.rows(prob, L, B, T)
        elapsed = time.perf_counter() - t0
    # target rows per second -> source tokens per second (T_s / T_t source tokens per row)
    src_per_row = spec.src_tokens * spec.batch / float(prob.tgt_tokens.sum())
    return {"value": passes * n_tok * src_per_row / elapsed, "unit": "tokens/s",
            "cores": O.num_threads(), "kind": "oracle",
            "sample": f"{passes} pass(es) over {n_tok} target tokens x all {lt} target layers "
                      f"(K and V), fp64 C oracle, {elapsed:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle-s", type=float, default=0.5,
                    help="seconds of untimed calls before the warm-up, so the GPU clocks "
                         "reach their loaded steady state")
    ap.add_argument("--config", type=int, default=2, help="workload 1-5 (default 2)")
    ap.add_argument("--tokens", type=int, default=None, help="override source tokens")
    ap.add_argument("--batch", type=int, default=None, help="override contexts per call")
    ap.add_argument("--sets", type=int, default=3, help="rotating buffer sets")
    ap.add_argument("--precision", choices=["bf16x2", "bf16", "f16", "bf16x2o"], default="bf16x2",
                    help="operand precision; bf16x2o splits only the k-steps holding the "
                         "workload's outlier channels")
    ap.add_argument("--paged", type=int, default=0, metavar="BLOCK",
                    help="write a paged target cache with BLOCK tokens per block through a "
                         "shuffled block table (0 = contiguous target layout)")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--fit", action="store_true",
                    help="measure the translator fit (accumulate + solve) instead")
    ap.add_argument("--lam", type=float, default=1.0, help="ridge of the fit's solve")
    ap.add_argument("--staged", action="store_true",
                    help="measure the staged (three-launch) translation stage by stage, "
                         "beside the fused kernel, instead")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first run a plain device copy (bitwise_not) of this many MiB "
                         "(three times), "
                         "a known-size reference for the HBM byte counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the translation would shard by target "
              "layer with no exchange, but this benchmark has no multi-GPU mode "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_30963_amd import kvx, synth as S

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    kvx.load()  # fails loudly if the library is not built

    spec = S.config(args.config, src_tokens=args.tokens, batch=args.batch)
    print(f"[bench] generating {spec.name} T={spec.src_tokens} B={spec.batch}",
          file=sys.stderr, flush=True)
    prob = S.make_problem(spec)
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib << 20
        csrc = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        cdst = torch.empty_like(csrc)
        torch.cuda.synchronize()
        for _ in range(3):  # an elementwise kernel: reads n bytes, writes n bytes
            torch.bitwise_not(csrc, out=cdst)
        torch.cuda.synchronize()
        del csrc, cdst
    if args.fit:
        return main_fit(args, spec, prob, torch, kvx, S)
    if args.staged:
        return main_staged(args, spec, prob, torch, kvx, S)
    alg = algorithmic(spec, prob)

    def dev(a, f32=False):
        if a is None:
            return None
        if spec.dtype == "bf16" and a.dtype == np.uint16 and not f32:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    kd = kvx.KVX_BF16 if spec.dtype == "bf16" else kvx.KVX_F32
    prec = {"bf16x2": kvx.KVX_PREC_BF16X2, "bf16": kvx.KVX_PREC_BF16,
            "f16": kvx.KVX_PREC_F16, "bf16x2o": kvx.KVX_PREC_BF16X2_OUTLIER}[args.precision]
    w_k, w_v = dev(prob.w_k), dev(prob.w_v)
    marks = {}
    if prec == kvx.KVX_PREC_BF16X2_OUTLIER:
        marks = {"outlier_k": S.outlier_channels(spec, 0), "outlier_v": S.outlier_channels(spec, 1)}
    tr = kvx.Translator(spec.src, spec.tgt, spec.mix, spec.layer_map, kd, w_k, w_v,
                        dev(prob.b_k), dev(prob.b_v), prec, **marks)
    del w_k, w_v
    info = tr.info()
    ident = prob.row_ptr is None
    rp, ci, wt = (None, None, None) if ident else (dev(prob.row_ptr), dev(prob.col_idx),
                                                  dev(prob.weight))
    cap = prob.tgt_capacity
    tdt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    oshape = (spec.tgt.n_layers, spec.batch, spec.tgt.n_kv_heads, cap, spec.tgt.head_dim)
    bt_dev, paging = None, {}
    if args.paged > 0:
        # every context's logical blocks on distinct, shuffled physical blocks
        bs = args.paged
        need = [(int(t) + bs - 1) // bs for t in prob.tgt_tokens]
        nblk = sum(need)
        perm = np.random.default_rng(0).permutation(nblk).astype(np.int32)
        table = np.zeros((spec.batch, max(need)), dtype=np.int32)
        k = 0
        for b, n in enumerate(need):
            table[b, :n] = perm[k:k + n]
            k += n
        bt_dev = torch.from_numpy(table).cuda()
        oshape = (spec.tgt.n_layers, nblk, spec.tgt.n_kv_heads, bs, spec.tgt.head_dim)
        paging = {"block_table": bt_dev, "block_size": bs, "max_blocks": table.shape[1],
                  "num_blocks": nblk}
    sk0, sv0 = dev(prob.src_k), dev(prob.src_v)
    sets = []
    for i in range(max(1, args.sets)):
        sk = sk0 if i == 0 else sk0.clone()
        sv = sv0 if i == 0 else sv0.clone()
        tk = torch.empty(oshape, dtype=tdt, device="cuda")
        tv = torch.empty(oshape, dtype=tdt, device="cuda")
        sets.append((sk, sv, tk, tv))
    tt = None if ident else prob.tgt_tokens
    stream = torch.cuda.current_stream()
    ios = [kvx.make_io(spec.batch, spec.src_tokens, s[0], s[1], s[2], s[3], cap, tt, rp, ci,
                       wt, **paging) for s in sets]

    def step(i):
        kvx.kvx_translate(tr.plan, ios[i % len(ios)][0], stream)

    # Clock settling: the GPU raises its clocks only after some time under
    # load (a 50-step run measured right after 5 warm-up calls is ~20% slower
    # than the steady state), so the workload first runs for settle_s seconds
    # of wall time; then come the W warm-up calls and the K timed ones.
    settle_calls = 0
    t_settle0 = time.perf_counter()
    while time.perf_counter() - t_settle0 < args.settle_s:
        for _ in range(20):
            step(settle_calls)
            settle_calls += 1
        torch.cuda.synchronize()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print(f"[bench] settled ({settle_calls} calls), warmup done ({args.warmup} calls); "
          f"timing {args.steps}", file=sys.stderr, flush=True)

    # Events on the stream the kernel is launched on: one pair around each
    # call (each call is one kernel launch), so the kernel's own average
    # duration is measured beside the whole timed region.
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    for i in range(args.steps):
        evs[i][0].record(stream)
        step(i)
        evs[i][1].record(stream)
    clock = gpu_clock_mhz()  # sampled while the enqueued calls run
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall0
    ms_ev = evs[0][0].elapsed_time(evs[-1][1]) / args.steps
    launch_ms = np.array([e0.elapsed_time(e1) for e0, e1 in evs])
    ms_kernel = float(launch_ms.mean())
    ms_wall = t_wall * 1e3 / args.steps
    ms = max(ms_ev, 0.0)

    # one more call per set, checked for unwritten rows (targets start uninitialised,
    # so fill with NaN first)
    for s in sets:
        s[2].fill_(float("nan"))
        s[3].fill_(float("nan"))
    for i in range(len(sets)):
        step(i)
    torch.cuda.synchronize()
    for s in sets:
        if args.paged > 0:  # every block of the table is fully used except tails
            unwritten = int(torch.isnan(s[2]).sum() + torch.isnan(s[3]).sum())
            tail = sum(-int(t) % args.paged for t in prob.tgt_tokens)
            bad = unwritten != 2 * tail * spec.tgt.n_layers * spec.tgt.n_kv_heads * \
                spec.tgt.head_dim
        else:
            bad = any(torch.isnan(s[2][:, b, :, :int(t)]).any() or
                      torch.isnan(s[3][:, b, :, :int(t)]).any()
                      for b, t in enumerate(prob.tgt_tokens))
        if bad:
            print("bench.py: output has unwritten rows", file=sys.stderr)
            sys.exit(1)

    tokens = spec.batch * spec.src_tokens
    value = tokens / (ms * 1e-3)
    # roofline of the kernel: algorithmic bytes (flops) per launch over the
    # kernel's average launch duration
    gbs = alg["bytes"] / (ms_kernel * 1e-3) / 1e9
    tfs = alg["flops"] / (ms_kernel * 1e-3) / 1e12
    kernel_name = "fused_kernel" if info.kernel == 1 else "tiled_kernel"
    layout = f"paged, {args.paged}-token blocks" if args.paged else "contiguous"
    traffic = recorded_traffic(spec.name, args.precision, spec.src_tokens, spec.batch, layout)
    busy = recorded(spec.name, args.precision, spec.src_tokens, spec.batch, layout,
                    "mfma_busy_frac")
    roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": kernel_name,
            "bytes_per_launch": alg["bytes"], "ms_per_launch": round(ms_kernel, 5),
            "mfma_tflops": round(tfs, 1),
            "mfma_frac": round(tfs / MFMA_BF16_PEAK_TFS, 4),
            # counter-based: share of the kernel's cycles its SIMDs' matrix
            # cores were busy (split operands issue more MFMAs than the
            # algorithmic contraction counts), from the committed summary
            "mfma_busy_frac": None if busy is None else float(busy)}

    cpu = None
    if not args.no_cpu and args.cpu_budget > 0:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cpu = cpu_baseline(spec, prob, args.cpu_budget)

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "settle_calls": settle_calls,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": spec.dtype, "data": "synthetic",
        "config": {"workload": spec.name, "src_tokens": spec.src_tokens,
                   "tgt_tokens": int(prob.tgt_tokens.sum()), "batch": spec.batch,
                   "src_layers": spec.src.n_layers, "tgt_layers": spec.tgt.n_layers,
                   "src_heads": f"{spec.src.n_kv_heads}x{spec.src.head_dim}",
                   "tgt_heads": f"{spec.tgt.n_kv_heads}x{spec.tgt.head_dim}",
                   "mix": spec.mix, "precision": args.precision,
                   "target_layout": layout,
                   "parallelism": "single GPU"},
        "ms_per_handoff": round(ms, 5) if spec.batch == 1 else None,
        "ms_wall_per_step": round(ms_wall, 5),
        # spread of the per-launch durations (HIP events around each call)
        "launch_ms_p10_p50_p90": [round(float(np.percentile(launch_ms, q)), 5)
                                  for q in (10, 50, 90)],
        "gpu_clock_mhz": clock,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    tr.close()


def staged_bytes(spec, prob, prec_split: bool):
    """Bytes each launch of the staged translation moves (one pass over all
    target layers): the algorithmic source, map, weight and target bytes of
    the operator, plus the intermediates as the stages write and read them
    (Z: bf16 planes, rows rounded up to 128 per context; U: fp32)."""
    alg = algorithmic(spec, prob)
    lt, din, dout = spec.tgt.n_layers, spec.d_in, spec.d_out
    rows_p = int(sum((int(t) + 127) // 128 * 128 for t in prob.tgt_tokens))
    ident = prob.row_ptr is None
    planes = [2 if prec_split else 1, 2 if prec_split and not ident else 1]
    z = sum(lt * p * rows_p * din * 2 for p in planes)
    u = 2 * lt * rows_p * dout * 4
    bias = 2 * lt * dout * 4
    return {"pool": alg["read"] + alg["map"] + z, "project": z + alg["weights"] + u,
            "store": u + bias + alg["write"], "z": z, "u": u,
            "flops_issued": 2 * lt * rows_p * din * dout * sum(planes)}


def main_staged(args, spec, prob, torch, kvx, S):
    """Per-stage time and memory throughput of kvx_translate_staged (pool,
    project, store: one launch each over all target layers), with the fused
    kernel timed on the same buffers for comparison."""
    if spec.dtype != "bf16" or args.paged:
        print("bench.py --staged: bf16 workloads, contiguous target layout", file=sys.stderr)
        sys.exit(2)
    prec = {"bf16x2": kvx.KVX_PREC_BF16X2, "bf16": kvx.KVX_PREC_BF16}.get(args.precision)
    if prec is None:
        print("bench.py --staged: precision bf16x2 or bf16", file=sys.stderr)
        sys.exit(2)

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    tr = kvx.Translator(spec.src, spec.tgt, spec.mix, spec.layer_map, kvx.KVX_BF16,
                        dev(prob.w_k), dev(prob.w_v), dev(prob.b_k), dev(prob.b_v), prec)
    ident = prob.row_ptr is None
    rp, ci, wt = (None, None, None) if ident else (dev(prob.row_ptr), dev(prob.col_idx),
                                                  dev(prob.weight))
    cap = prob.tgt_capacity
    oshape = (spec.tgt.n_layers, spec.batch, spec.tgt.n_kv_heads, cap, spec.tgt.head_dim)
    sk, sv = dev(prob.src_k), dev(prob.src_v)
    tk = torch.full(oshape, float("nan"), dtype=torch.bfloat16, device="cuda")
    tv = torch.full(oshape, float("nan"), dtype=torch.bfloat16, device="cuda")
    io, keep = kvx.make_io(spec.batch, spec.src_tokens, sk, sv, tk, tv, cap,
                           None if ident else prob.tgt_tokens, rp, ci, wt)
    nws = kvx.kvx_staged_workspace_bytes(tr.plan, io, spec.tgt.n_layers)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    stages = [("pool", kvx.KVX_STAGE_POOL), ("project", kvx.KVX_STAGE_PROJECT),
              ("store", kvx.KVX_STAGE_STORE)]

    def staged_step():
        for _, m in stages:
            kvx.kvx_translate_staged(tr.plan, io, ws, stages=m, stream=stream)

    t0 = time.perf_counter()
    calls = 0
    while time.perf_counter() - t0 < args.settle_s:
        staged_step()
        kvx.kvx_translate(tr.plan, io, stream)
        calls += 1
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        staged_step()
    torch.cuda.synchronize()
    if any(torch.isnan(x[:, b, :, :int(t)]).any() for x in (tk, tv)
           for b, t in enumerate(prob.tgt_tokens)):
        print("bench.py: staged output has unwritten rows", file=sys.stderr)
        sys.exit(1)
    # events on the launch stream around every stage launch
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in stages] for _ in range(args.steps)]
    evf = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        for j, (_, m) in enumerate(stages):
            ev[i][j][0].record(stream)
            kvx.kvx_translate_staged(tr.plan, io, ws, stages=m, stream=stream)
            ev[i][j][1].record(stream)
    for i in range(args.steps):
        evf[i][0].record(stream)
        kvx.kvx_translate(tr.plan, io, stream)
        evf[i][1].record(stream)
    torch.cuda.synchronize()
    ms_stage = [sum(ev[i][j][0].elapsed_time(ev[i][j][1]) for i in range(args.steps)) / args.steps
                for j in range(len(stages))]
    ms_fused = sum(a.elapsed_time(b) for a, b in evf) / args.steps
    by = staged_bytes(spec, prob, prec == kvx.KVX_PREC_BF16X2)
    alg = algorithmic(spec, prob)
    per = {}
    for (name, _), ms in zip(stages, ms_stage):
        gbs = by[name] / (ms * 1e-3) / 1e9
        per[name] = {"ms": round(ms, 5), "bytes": by[name], "gbs": round(gbs, 1),
                     "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
    tfs = by["flops_issued"] / (ms_stage[1] * 1e-3) / 1e12
    per["project"]["mfma_tflops_issued"] = round(tfs, 1)
    per["project"]["mfma_frac_issued"] = round(tfs / MFMA_BF16_PEAK_TFS, 4)
    total = sum(ms_stage)
    tokens = spec.batch * spec.src_tokens
    out = {
        "metric": "staged translation: per-stage ms and GB/s (pool, project, store) beside "
                  "the fused kernel",
        "value": round(tokens / (total * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(total, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": spec.name, "src_tokens": spec.src_tokens,
                   "tgt_tokens": int(prob.tgt_tokens.sum()), "batch": spec.batch,
                   "precision": args.precision, "parallelism": "single GPU"},
        "stages": per,
        "fused": {"ms": round(ms_fused, 5), "bytes": alg["bytes"],
                  "gbs": round(alg["bytes"] / (ms_fused * 1e-3) / 1e9, 1)},
        "staged_over_fused": round(total / ms_fused, 3),
        "workspace_bytes": nws,
    }
    print(json.dumps(out), flush=True)
    del keep
    tr.close()


def fit_flops(spec, rows: int, fit_bias: bool = True) -> int:
    """Algorithmic flops of accumulating `rows` rows: per (layer, K|V) system
    the symmetric Zt^T Zt (n(n+1)/2 entries) and Zt^T Y, 2 flops per term."""
    n = spec.d_in + (1 if fit_bias else 0)
    return 2 * spec.tgt.n_layers * 2 * rows * (n * (n + 1) // 2 + n * spec.d_out)


def fit_issued_flops(spec, prob, rows: int) -> int:
    """Matrix-core flops fit_gram issues for `rows` rows: 128 x 128 blocks
    (bi over the Z features, bj >= bi over Z and Y, padded), rows padded to
    64, and per block the products hi*hi (+ hi*lo, lo*hi for operands that are
    not exact bf16: computed ones, or fp32 data)."""
    bf = spec.dtype == "bf16"
    ident = prob.row_ptr is None
    nbz = -(-spec.d_in // 128)
    nbj = nbz + -(-spec.d_out // 128)
    rows_p = -(-rows // 64) * 64
    total = 0
    for kv in (0, 1):
        lo_z = not (bf and ident and (kv == 1 or spec.src.rope_base <= 0))
        lo_y = not (bf and (kv == 1 or spec.tgt.rope_base <= 0))
        for bi in range(nbz):
            for bj in range(bi, nbj):
                total += 1 + lo_z + (lo_z if bj < nbz else lo_y)
    return 2 * 128 * 128 * rows_p * total * spec.tgt.n_layers


def fit_cpu_baseline(spec, prob, tk, tv, lam: float, budget_s: float):
    """The fp64 fit oracle on the host over as many target layers as fit the
    budget (all rows, K and V), scaled to rows per second of the whole job."""
    from oracle import fit as F
    import dataclasses
    rows = int(prob.tgt_tokens.sum())
    done, t0 = 0, time.perf_counter()
    for l in range(spec.tgt.n_layers):
        sub = dataclasses.replace(spec, tgt=dataclasses.replace(spec.tgt, n_layers=1),
                                  layer_map=tuple(spec.layer_map[l * spec.mix:(l + 1) * spec.mix]))
        p1 = dataclasses.replace(prob, spec=sub, layer_map=np.asarray(sub.layer_map, np.int32))
        F.fit(p1, tk[l:l + 1], tv[l:l + 1], lam, True)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": rows * done / spec.tgt.n_layers / el, "unit": "rows/s",
            "cores": os.cpu_count(), "kind": "oracle",
            "sample": f"fp64 numpy fit oracle, {done} of {spec.tgt.n_layers} target layers "
                      f"(K and V, all {rows} rows), {el:.1f} s"}


def main_fit(args, spec, prob, torch, kvx, S):
    os.environ["KVX_FIT_TIMING"] = "1"
    kd = kvx.KVX_BF16 if spec.dtype == "bf16" else kvx.KVX_F32
    print("[bench] drawing native target caches", file=sys.stderr, flush=True)
    tk = S.draw_native_target(spec, 0, prob.tgt_tokens)
    tv = S.draw_native_target(spec, 1, prob.tgt_tokens)

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    sk, sv, dk, dv = dev(prob.src_k), dev(prob.src_v), dev(tk), dev(tv)
    ident = prob.row_ptr is None
    rp, ci, wt = (None, None, None) if ident else (dev(prob.row_ptr), dev(prob.col_idx),
                                                  dev(prob.weight))
    tt = None if ident else prob.tgt_tokens
    fitter = kvx.Fitter(spec.src, spec.tgt, spec.mix, spec.layer_map, kd, True)
    stream = torch.cuda.current_stream()

    def step():
        fitter.accumulate(sk, sv, dk, dv, tt, rp, ci, wt, stream=stream)

    settle_calls = 0
    t_settle0 = time.perf_counter()
    while time.perf_counter() - t_settle0 < args.settle_s:  # clock settling, as above
        step()
        settle_calls += 1
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    fitter.info()            # drop the warm-up launches' timing events
    fitter.reset()
    print(f"[bench] fit warmup done; timing {args.steps} accumulates", file=sys.stderr,
          flush=True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    info = fitter.info()
    # one Gram pass per layer group and step: the K-system and the V-system
    # launch, timed together
    ms_gram = info.gram_ms / max(1, info.gram_launches)
    passes_per_step = info.gram_launches / args.steps
    rows = int(prob.tgt_tokens.sum())
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record(stream)
    w_k, w_v, b_k, b_v = fitter.solve(args.lam, stream=stream)
    s1.record(stream)
    torch.cuda.synchronize()
    ms_solve = s0.elapsed_time(s1)
    if not (torch.isfinite(w_k).all() and torch.isfinite(w_v).all()):
        print("bench.py: fit produced non-finite weights", file=sys.stderr)
        sys.exit(1)
    flops_step = fit_flops(spec, rows)
    flops_pass = flops_step / passes_per_step
    tfs = flops_pass / (ms_gram * 1e-3) / 1e12
    cpu = None
    if not args.no_cpu and args.cpu_budget > 0:
        print("[bench] timing the CPU fit oracle", file=sys.stderr, flush=True)
        cpu = fit_cpu_baseline(spec, prob, tk, tv, args.lam, args.cpu_budget)
    out = {
        "metric": "fit rows/s (paired target tokens accumulated into every layer's K and V "
                  "normal equations)",
        "value": round(rows / (ms * 1e-3), 1), "unit": "rows/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "settle_calls": settle_calls,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16x2->fp32 accumulate, fp64 solve", "data": "synthetic",
        "config": {"workload": f"translator fit, {spec.name}", "rows": rows,
                   "src_tokens": spec.src_tokens, "batch": spec.batch,
                   "systems": info.systems, "unknowns": info.n, "outputs": spec.d_out,
                   "lambda": args.lam, "parallelism": "single GPU"},
        "ms_per_solve": round(ms_solve, 3),
        "roofline": {"bound": "mfma", "achieved": round(tfs, 1), "peak": MFMA_BF16_PEAK_TFS,
                     "unit": "TFLOP/s", "frac": round(tfs / MFMA_BF16_PEAK_TFS, 4),
                     "traffic": None, "kernel": "fit_gram (K and V launches of a pass)",
                     "flops_per_pass": int(flops_pass), "ms_per_pass": round(ms_gram, 5),
                     "issued_mfma_flops_per_pass": int(
                         fit_issued_flops(spec, prob, rows) / passes_per_step)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    fitter.close()


if __name__ == "__main__":
    main()
