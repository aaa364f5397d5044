#!/usr/bin/env python3
"""Useful document-masked attention TFLOP/s for one sequence-parallel shard on one MI355X.

One step is one pass of the whole path for one packed batch, inputs resident
in HBM, driven by the step executor (hsap_executor_*):
  host planner (tile list and runs, C++) -> one async upload of the lists
  -> partial attention of the shard against every K/V chunk -> LSE merge
  (and, for a forward+backward workload, the document starts, the backward
  preprocess and the partial attention backward, which stores the final bf16
  dQ/dK/dV from its registers).

Timing: about 60 ms of untimed steps first (the GPU's clocks settle under
sustained load), then the warm-up steps, then the timed steps with nothing
between the launches; a second pass of the same steps with events around
each stage gives the per-kernel breakdown.

Default workload: the largest single-GPU configuration, a 262144-token packed
sequence with Pareto document lengths, head-parallel degree 4 x ring degree 8
(contiguous): the shard holds 8 of 32 heads of 128 and 1/8 of the tokens, shard
4 (the one with the most allowed pairs), forward.  The other workloads are
reported under "extra", each with its own roofline figures; a name with "+bwd"
runs that workload forward + backward.

Prints ONE JSON line on stdout; progress goes to stderr.
  python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload c4]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
SETTLE_S = 0.06             # untimed sustained load before the warm-up steps (clocks reach steady state)
SETTLE_MAX_STEPS = 4000
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "useful doc-masked attention TFLOP/s per shard; % of bf16 MFMA peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _critical_shard(L, w):
    best, best_r = -1, 0
    for r in range(w.sp_degree):
        d = L.shard_desc(w.total_tokens, w.sp_degree, w.layout, r, w.block_m, w.block_n, batch=w.batch)
        pairs = int(L.plan(w.cu_seqlens, d)["useful_pairs"].sum())
        if pairs > best:
            best, best_r = pairs, r
    return best_r


def _positions(N: int, P: int, layout: int, x: int, local: np.ndarray) -> np.ndarray:
    """Global positions of local rows of shard (or chunk) x; row b*n + l is row l of sequence b of
    N tokens (a batch of concatenated sequences)."""
    n = N // P
    b, local = local // n, local % n
    if layout == 0:
        return b * N + x * n + local
    m = n // 2
    return b * N + np.where(local < m, x * m + local, (2 * P - 1 - x) * m + (local - m))


def _merged_rows(L, cu, sd, split: int):
    """(finite, merged): the (part, query row) pairs whose partial LSE is finite among the rows the
    merge handles, and the number of those rows, from the plan on the host.  A q-tile whose only
    run holding tiles is unsplit is written final by the partial forward and not merged; a row of a
    q-major run has an allowed key iff some tile of the run holds a key j with start(i) <= j <= i."""
    tiles = L.plan(cu, sd)["tiles"]
    sorted_tiles, runs, _ = L.plan_runs(sd, tiles, L.MAJOR_Q, split)
    N, P, bm, bn = sd.total_tokens, sd.sp_degree, sd.block_m, sd.block_n
    busy = np.bincount(runs[runs[:, 3] > 0][:, 1], minlength=sd.rows // bm)
    starts = np.repeat(cu[:-1].astype(np.int64), np.diff(cu))
    count = 0
    for _, t, first, cnt in runs:
        if cnt == 0 or busy[t] == 1:
            continue
        gi = _positions(N, P, sd.layout, sd.shard_id, np.arange(t * bm, (t + 1) * bm))
        si = starts[gi]
        ok = np.zeros(bm, dtype=bool)
        for c, _, kt, _ in sorted_tiles[first:first + cnt]:
            k0 = int(_positions(N, P, sd.layout, int(c), np.array([kt * bn]))[0])  # a tile's keys are contiguous
            ok |= (k0 <= gi) & (k0 + bn - 1 >= si)
        count += int(ok.sum())
    return count, int(np.sum(busy != 1)) * bm


def measure(name: str, steps: int, warmup: int, backward=None):
    """Time `steps` steps of one workload through the step executor; returns a result dict (GPU side only).
    A name ending in "+bwd" runs the workload forward + backward."""
    import torch
    from paper_2606_30460_amd import _lib as L
    from paper_2606_30460_amd.shard_attention import to_sharded
    from workloads import make_workload

    if name.endswith("+bwd"):
        name, backward = name[:-4], True
    w = make_workload(name)
    bwd = w.backward if backward is None else backward
    shard = w.shard if w.shard is not None else _critical_shard(L, w)
    log("[bench] %s: generating inputs (shard %d)" % (w.name, shard))
    t = w.tensors(backward=bwd)
    dev = torch.device("cuda")
    sd = L.shard_desc(w.total_tokens, w.sp_degree, w.layout, shard, w.block_m, w.block_n, batch=w.batch)
    desc = L.attn_desc(sd, w.heads_q, w.heads_kv, w.head_dim, 1.0 / math.sqrt(w.head_dim))
    # the step's executor plans only the lists the step reads (the fused forward's lists are planned
    # and uploaded by a second executor, timed apart below)
    ex = L.Executor(desc, backward=bwd)
    q = to_sharded(sd, t["q"].to(dev))[shard].contiguous()
    k = to_sharded(sd, t["k"].to(dev))
    v = to_sharded(sd, t["v"].to(dev))
    d_o = to_sharded(sd, t["do"].to(dev))[shard].contiguous() if bwd else None
    del t
    n = sd.rows
    o = torch.empty(n, w.heads_q, w.head_dim, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(w.heads_q, n, dtype=torch.float32, device=dev)
    if bwd:
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    cu = np.ascontiguousarray(w.cu_seqlens, dtype=np.int32)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()

    def one_step(e):
        # a training step re-plans its batch: host planner, one upload, document starts
        ex.plan(cu)
        if e:
            e[0].record()
        ex.partial_forward(q, k, v, o, lse)
        if e:
            e[1].record()
        ex.merge(o, lse)
        if e:
            e[2].record()
        if bwd:
            ex.backward(q, k, v, d_o, o, lse, dq, dk, dv)
            if e:
                e[3].record()

    # Settle: under sustained load the GPU's clocks take some tens of milliseconds to reach their
    # steady state (the first ~150 c2 steps run up to a third slower than the later ones, which a
    # training job never sees after its first moments).  Run the same step untimed for about
    # SETTLE_S, in bursts of 10 with a synchronisation between bursts, then the warm-up steps.
    settle_steps, t_settle = 0, time.perf_counter()
    while time.perf_counter() - t_settle < SETTLE_S and settle_steps < SETTLE_MAX_STEPS:
        for _ in range(10):
            one_step(None)
        settle_steps += 10
        torch.cuda.synchronize()
    for _ in range(warmup):
        one_step(None)
    torch.cuda.synchronize()
    # the step rate, timed with nothing between the launches; then the same steps again with
    # events around each stage for the per-kernel breakdown (event markers add small gaps)
    t0 = time.perf_counter()
    for i in range(steps):
        one_step(None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for i in range(steps):
        one_step(events[i])
    torch.cuda.synchronize()
    info = ex.info()

    fwd_ms = np.array([e[0].elapsed_time(e[1]) for e in events])
    merge_ms = np.array([e[1].elapsed_time(e[2]) for e in events])
    bwd_ms = np.array([e[2].elapsed_time(e[3]) for e in events]) if bwd else None

    # the fused forward (partials and merge in one pass), same plan and inputs, launches back to back
    fused_ms = None
    if not bwd:
        fo, fl = torch.empty_like(o), torch.empty_like(lse)
        exf = L.Executor(desc, fused=True)
        exf.plan(cu)
        for _ in range(3):
            exf.forward(q, k, v, fo, fl, fused=True)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(steps):
            exf.forward(q, k, v, fo, fl, fused=True)
        ev[1].record()
        torch.cuda.synchronize()
        fused_ms = ev[0].elapsed_time(ev[1]) / steps
        exf.close()

    # planner host time alone (hsap_plan; overlapped with the GPU inside a step)
    t1 = time.perf_counter()
    reps = 20
    for _ in range(reps):
        L.plan(cu, sd)
    plan_ms = (time.perf_counter() - t1) / reps * 1e3

    # algorithmic merge bytes over the rows it merges: every part's LSE, the O rows of parts whose
    # LSE is finite, the outputs (rows of single-part q-tiles are written final by the forward)
    finite, merged = _merged_rows(L, cu, sd, info["split_length"])
    merge_bytes = (info["num_parts"] * w.heads_q * merged * 4 + finite * w.heads_q * w.head_dim * 4
                   + merged * w.heads_q * (2 * w.head_dim + 4))

    pairs = info["useful_pairs"]
    tiles = info["num_tiles"]
    fwd_flops = 4.0 * w.head_dim * w.heads_q * pairs
    bwd_flops = 10.0 * w.head_dim * w.heads_q * pairs if bwd else 0.0
    ms_step = wall / steps * 1e3
    res = {
        "workload": w.name, "workload_key": name, "shard": shard, "tokens": w.total_tokens, "batch": w.batch, "sp_degree": w.sp_degree,
        "layout": w.layout, "heads_q": w.heads_q, "heads_kv": w.heads_kv, "head_dim": w.head_dim,
        "block_m": w.block_m, "block_n": w.block_n, "backward": bool(bwd), "docs": w.num_docs,
        "useful_pairs": pairs, "tiles": tiles, "full_tiles": info["num_full_tiles"],
        "tile_efficiency": pairs / float(tiles * w.block_m * w.block_n),
        "chunks_with_tiles": info["chunks_with_tiles"],
        "partial_slots": info["num_parts"], "split_length": info["split_length"],
        "useful_gflop_per_step": (fwd_flops + bwd_flops) / 1e9,
        "ms_per_step": ms_step,
        "tflops": (fwd_flops + bwd_flops) / (ms_step * 1e-3) / 1e12,
        "fwd_kernel_ms_mean": float(fwd_ms.mean()), "fwd_kernel_ms_median": float(np.median(fwd_ms)),
        "fwd_kernel_ms_min": float(fwd_ms.min()),
        "fwd_kernel_tflops": fwd_flops / (fwd_ms.mean() * 1e-3) / 1e12,
        "merge_kernel_ms_mean": float(merge_ms.mean()),
        "merge_bytes": merge_bytes,
        "merge_gbs": merge_bytes / (merge_ms.mean() * 1e-3) / 1e9,
        "planner_host_ms": plan_ms,
        "settle_steps": settle_steps,
    }
    if fused_ms is not None:
        res.update({"fused_fwd_kernel_ms": fused_ms, "fused_fwd_tflops": fwd_flops / (fused_ms * 1e-3) / 1e12})
    if bwd:
        res.update({"bwd_ms_mean": float(bwd_ms.mean()), "bwd_ms_median": float(np.median(bwd_ms)),
                    "bwd_tflops": bwd_flops / (bwd_ms.mean() * 1e-3) / 1e12})
    # the dominant kernel's roofline figures: useful flops of one launch over its mean duration
    fwd_achieved = fwd_flops / (fwd_ms.mean() * 1e-3) / 1e12
    res["roofline"] = {"bound": "mfma", "kernel": fwd_kernel_name(res), "achieved": round(fwd_achieved, 3),
                       "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(fwd_achieved / PEAK_BF16_TFLOPS, 5)}
    if bwd:
        bwd_achieved = bwd_flops / (bwd_ms.mean() * 1e-3) / 1e12
        res["roofline_bwd"] = {"bound": "mfma", "kernels": bwd_kernel_names(res), "achieved": round(bwd_achieved, 3),
                               "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                               "frac": round(bwd_achieved / PEAK_BF16_TFLOPS, 5)}
    res["_fwd_flops"] = fwd_flops
    log("[bench] %s: %.3f ms/step, %.1f TFLOP/s useful (fwd kernel %.3f ms = %.1f TFLOP/s)" % (
        w.name, ms_step, res["tflops"], res["fwd_kernel_ms_mean"], res["fwd_kernel_tflops"]))
    ex.close()
    del q, k, v, o, lse
    torch.cuda.empty_cache()
    return res


def cpu_baseline(name: str, budget_s: float):
    """The fp64 oracle on a bounded sample of the workload's query rows, on the host cores."""
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    from workloads import make_workload
    from paper_2606_30460_amd import _lib as L

    w = make_workload(name)
    shard = w.shard if w.shard is not None else _critical_shard(L, w)
    t = w.tensors(backward=False)
    q, k, v = (t[x].float().numpy() for x in ("q", "k", "v"))
    cores = len(os.sched_getaffinity(0))
    n = w.total_tokens // w.sp_degree
    pos_all = oracle.shard_positions(w.total_tokens, w.sp_degree, w.layout, shard)
    starts = oracle.doc_starts(w.cu_seqlens)
    rng = np.random.default_rng(0)
    with threadpool_limits(limits=cores):
        used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        # double the sample until one oracle run takes at least half the budget
        count = 64
        while True:
            count = min(count, n)
            rows = np.sort(rng.choice(n, size=count, replace=False))
            t0 = time.perf_counter()
            oracle.shard_forward(q, k, v, w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, shard, rows=rows)
            el = time.perf_counter() - t0
            log("[bench] oracle: %d rows in %.1f s" % (count, el))
            if el >= 0.5 * budget_s or count == n:
                break
            count *= 2
    pos = pos_all[rows]
    pairs = int(np.sum(pos - starts[pos] + 1))
    flops = 4.0 * w.head_dim * w.heads_q * pairs
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        cpu_model = platform.processor()
    return {"value": flops / el / 1e12, "unit": "TFLOP/s", "cores": int(used), "kind": "oracle",
            "sample": "%d of %d query rows of shard %d (all %d heads, all %d chunks, merge), fp64 numpy/BLAS, "
                      "%.1f s, %.2f useful GFLOP" % (count, n, shard, w.heads_q, w.sp_degree, el, flops / 1e9),
            "cpu": cpu_model, "affinity_cores": cores}


def all_shards_analysis(name: str, layouts=None, reps: int = 5) -> dict:
    """Every shard of the workload's packed sequence on this GPU, ring and balanced schedules
    (hsap_load_matrix, hsap_balance): per-rank tiles and milliseconds (blocks + merge, median of
    ``reps``), the critical path, and the whole sequence's useful TFLOP/s at that critical path,
    i.e. what a group of P GPUs would reach if each ran its rank's work alone, without transfers.
    The same assignment also runs as per-rank instruction lists (hsap_emit_forward) with every
    rank's stream on this one GPU: its stages, instruction count and wall time (all ranks' work
    plus the transfers as device copies, on one GPU)."""
    import torch
    from paper_2606_30460_amd import _lib as L
    from paper_2606_30460_amd.all_shards import AllShards
    from paper_2606_30460_amd.sap_program import SapProgram
    from paper_2606_30460_amd.shard_attention import to_sharded
    from workloads import make_workload, random_bf16

    w = make_workload(name)
    dev = torch.device("cuda")
    N, P = w.total_tokens, w.sp_degree
    q = random_bf16((N, w.heads_q, w.head_dim), w.seed + 1).to(dev)
    k = random_bf16((N, w.heads_kv, w.head_dim), w.seed + 2).to(dev)
    v = random_bf16((N, w.heads_kv, w.head_dim), w.seed + 3).to(dev)
    lengths = np.diff(w.cu_seqlens).astype(np.int64)
    flops = 4.0 * w.head_dim * w.heads_q * float(np.sum(lengths * (lengths + 1) // 2))
    out = {}
    for layout in (layouts or [w.layout]):
        s = L.shard_desc(N, P, layout, 0, w.block_m, w.block_n)
        qs, ks, vs = to_sharded(s, q), to_sharded(s, k), to_sharded(s, v)
        res = {}
        for balanced in (False, True):
            a = AllShards(w.cu_seqlens, N, P, layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n,
                          balance=balanced)
            a.plan()
            bufs = a.alloc()
            for _ in range(2):
                a.forward(qs, ks, vs, bufs)
            times = [a.forward(qs, ks, vs, bufs, timed=True) for _ in range(reps)]
            rank_ms = (np.median([t["blocks_ms"] for t in times], axis=0)
                       + np.median([t["merge_ms"] for t in times], axis=0))
            sched = a.schedule()
            crit = float(rank_ms.max())
            del bufs, a
            torch.cuda.empty_cache()
            # the same assignment as per-rank instruction lists (hsap_emit_forward), all ranks' streams on this GPU
            prog = SapProgram(w.cu_seqlens, N, P, layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n,
                              balance=balanced)
            prog.plan()
            pbufs = prog.alloc()
            prog.run(qs, ks, vs, pbufs)
            prog_ms = float(np.median([prog.run(qs, ks, vs, pbufs, timed=True) for _ in range(reps)]))
            n_ops = int(sum(len(x) for x in prog.ops))
            n_stages = prog.num_stages
            del pbufs, prog
            torch.cuda.empty_cache()
            res["balanced" if balanced else "ring"] = {
                "rank_tiles": sched["rank_tiles"], "tile_imbalance": round(sched["tile_imbalance"], 3),
                "moved_blocks": sched["moved_blocks"], "rank_ms": [round(x, 4) for x in rank_ms.tolist()],
                "critical_ms": round(crit, 4), "rank_ms_mean": round(float(rank_ms.mean()), 4),
                "sequence_tflops_at_critical_path": round(flops / (crit * 1e-3) / 1e12, 1),
                "kv_bytes_moved": sched["kv_bytes_moved"], "q_o_bytes_moved": sched["q_o_bytes_moved"],
                "program_stages": n_stages, "program_ops": n_ops, "program_one_gpu_ms": round(prog_ms, 4)}
        log("[bench] all shards %s %s: critical path ring %.3f ms, balanced %.3f ms" % (
            name, layout, res["ring"]["critical_ms"], res["balanced"]["critical_ms"]))
        out[layout] = res
    del q, k, v
    torch.cuda.empty_cache()
    return out


def fp8_analysis(name: str, reps: int = 50) -> dict:
    """The fp8 score variant on the workload's shard: e4m3 quantisation of Q and of every chunk's K
    (hsap_quantize_fp8), then the partial forward with fp8 scores (hsap_partial_attn_fwd_fp8) over
    the same plan as the bf16 partial forward, which is timed beside it; back-to-back launches
    between two events, mean per launch."""
    import torch
    from paper_2606_30460_amd import _lib as L
    from paper_2606_30460_amd.shard_attention import ShardAttention, to_sharded
    from workloads import make_workload

    w = make_workload(name)
    if w.head_dim != 128 or w.batch != 1:
        return {}
    shard = w.shard if w.shard is not None else _critical_shard(L, w)
    sa = ShardAttention(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, shard, w.heads_q, w.heads_kv,
                        w.head_dim, w.block_m, w.block_n)
    sa.plan()
    dev = torch.device("cuda")
    t = w.tensors(backward=False)
    q = to_sharded(sa.shard, t["q"].to(dev))[shard].contiguous()
    k, v = to_sharded(sa.shard, t["k"].to(dev)), to_sharded(sa.shard, t["v"].to(dev))
    del t
    q8 = torch.empty(q.shape, dtype=torch.uint8, device=dev)
    k8 = torch.empty(k.shape, dtype=torch.uint8, device=dev)
    qs = torch.empty(1, w.heads_q, dtype=torch.float32, device=dev)
    ks = torch.empty(w.sp_degree, w.heads_kv, dtype=torch.float32, device=dev)
    work = torch.empty(w.sp_degree * max(w.heads_q, w.heads_kv) * L.QUANT_SPLIT, dtype=torch.float32, device=dev)
    bufs = sa.alloc_forward()

    def timed(fn):  # about 30 ms of launches first (clocks settle under sustained load)
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.03:
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        for _ in range(reps):
            fn()
        e[1].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps

    wq, wk = work[:w.heads_q * L.QUANT_SPLIT], work[:w.sp_degree * w.heads_kv * L.QUANT_SPLIT]
    quant_ms = timed(lambda: (L.quantize_fp8(q.unsqueeze(0), q8.unsqueeze(0), qs, wq), L.quantize_fp8(k, k8, ks, wk)))
    fp8_ms = timed(lambda: L.partial_attn_fwd_fp8(sa.desc, q8, k8, v, qs, ks, sa.doc_start, sa.tiles_q, sa.runs_q,
                                                  bufs["o_part"], bufs["lse_part"]))
    bf16_ms = timed(lambda: L.partial_attn_fwd_runs(sa.desc, q, k, v, sa.doc_start, sa.tiles_q, sa.runs_q, bufs["o_part"],
                                               bufs["lse_part"]))
    flops = 4.0 * w.head_dim * w.heads_q * sa.total_useful_pairs
    log("[bench] fp8 scores %s: partial forward %.3f ms (%.1f TFLOP/s) vs bf16 %.3f ms; quantisation %.3f ms" % (
        name, fp8_ms, flops / (fp8_ms * 1e-3) / 1e12, bf16_ms, quant_ms))
    out = {"fp8_partial_fwd_ms": round(fp8_ms, 5), "fp8_partial_fwd_tflops": round(flops / (fp8_ms * 1e-3) / 1e12, 1),
           "bf16_partial_fwd_ms_same_loop": round(bf16_ms, 5),
           "bf16_partial_fwd_tflops_same_loop": round(flops / (bf16_ms * 1e-3) / 1e12, 1),
           "quantize_q_and_k_ms": round(quant_ms, 5)}
    del q, k, v, q8, k8, bufs, sa
    torch.cuda.empty_cache()
    return out


FWD_SOURCES = ("paper_2606_30460_amd/csrc/attn_fwd.hip", "paper_2606_30460_amd/csrc/mfma.h",
               "paper_2606_30460_amd/csrc/hsap_internal.h", "paper_2606_30460_amd/build.py")
TRAFFIC_GLOB = "profiles/attn_fwd_hbm_traffic*.md"


def fwd_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in FWD_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def fwd_kernel_name(res) -> str:
    """The partial forward kernel the library dispatches for a workload's shapes (bf16 scores):
    direct-to-LDS for head_dim 128 with 128- or 256-row q-tiles, register-staged otherwise."""
    d, bm, bn = res["head_dim"], res["block_m"], res["block_n"]
    if d == 128 and bm in (128, 256):
        return "attn_fwd_dl_kernel<%d, %d, false, false, false>" % (bn, bm // 32)
    return "attn_fwd_kernel<%d, %d, %d, false, false, false>" % (d, bn, bm // 32)


def bwd_kernel_names(res) -> list:
    """The two backward kernels the library dispatches for a workload's shapes (bf16 gradients)."""
    d, bm, bn = res["head_dim"], res["block_m"], res["block_n"]
    dkdv = ("attn_bwd_dkdv_split_kernel<true>" if d == 128 and bn == 128
            else "attn_bwd_dkdv_kernel<%d, %d, true, false>" % (d, bn // 32))
    return [dkdv, "attn_bwd_dq_kernel<%d, %d, %d, true, false>" % (d, bn, bm // 32)]


def measured_traffic(workload: str):
    """HBM bytes per forward launch from the committed counter summary of this workload, or None.

    Each summary (profiles/attn_fwd_hbm_traffic*.md) records the bytes measured with rocprofv3
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size) together with the workload and
    the hash of the forward kernel's sources at the time; a changed kernel reports None.
    """
    import glob
    for path in sorted(glob.glob(os.path.join(ROOT, TRAFFIC_GLOB))):
        fields = {}
        with open(path) as f:
            for line in f:
                if line.startswith("- ") and ":" in line:
                    k, v = line[2:].split(":", 1)
                    fields[k.strip()] = v.strip().strip("`")
        if fields.get("workload") != workload:
            continue
        if fields.get("kernel_source_sha256_16") != fwd_source_hash():
            return None
        try:
            return int(fields["hbm_bytes_per_launch"])
        except (KeyError, ValueError):
            return None
    return None


def calibrate_copy(nbytes: int) -> None:
    """A plain device-to-device copy of known size, for scaling HBM byte counters."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": src.numel() * 4, "copies": 3}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--extra", default="c2,c3,c5,c5m,c6,c3+bwd,c4+bwd",
                    help="other workloads reported under 'extra' ('' for none); 'name+bwd' runs forward + backward")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="oracle budget for the CPU baseline (0: skip)")
    ap.add_argument("--no-all-shards", action="store_true",
                    help="skip the all-shard load analysis of the main workload (e.g. under a kernel trace)")
    ap.add_argument("--all-shards", default="", metavar="WORKLOADS",
                    help="only run the all-shard load analysis (both layouts) of these workloads and print it")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the sequence-parallel split is simulated in memory on a single "
              "MI355X; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2606_30460_amd import _lib as L
    L.lib()
    if args.all_shards:
        print(json.dumps({name: all_shards_analysis(name, ["contiguous", "zigzag"])
                          for name in args.all_shards.split(",") if name}), flush=True)
        return

    main_res = measure(args.workload, args.steps, args.warmup)
    extra = {}
    for name in [x for x in args.extra.split(",") if x and x != args.workload]:
        r = measure(name, min(args.steps, 20), min(args.warmup, 3))
        r.pop("_fwd_flops", None)
        extra[name] = r
    if not args.no_all_shards:       # analyses beside the timed step, skipped under kernel traces
        for name, res in [(args.workload, main_res)] + list(extra.items()):
            if not res["backward"]:
                res["fp8_scores"] = fp8_analysis(res["workload_key"])
    if not args.no_all_shards:
        main_res["all_shards"] = all_shards_analysis(args.workload)
    cpu = None
    if args.cpu_seconds > 0:
        log("[bench] CPU baseline (oracle) on %s, ~%.0f s" % (args.workload, args.cpu_seconds))
        cpu = cpu_baseline(args.workload, args.cpu_seconds)

    main_res.pop("_fwd_flops")
    roof = dict(main_res["roofline"])
    roof.update({"traffic": measured_traffic(main_res["workload_key"]), "kernel_source_sha256_16": fwd_source_hash()})
    line = {
        "metric": METRIC,
        "value": round(main_res["tflops"], 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": main_res["workload"], "tokens": main_res["tokens"], "sp_degree": main_res["sp_degree"],
                   "layout": main_res["layout"], "shard": main_res["shard"], "heads_q": main_res["heads_q"],
                   "heads_kv": main_res["heads_kv"], "head_dim": main_res["head_dim"],
                   "block_m": main_res["block_m"], "block_n": main_res["block_n"], "pass": "forward"
                   if not main_res["backward"] else "forward+backward"},
        "pct_of_bf16_peak": round(100.0 * main_res["tflops"] / PEAK_BF16_TFLOPS, 3),
        "roofline": roof,
        "cpu_baseline": cpu,
        "detail": main_res,
        "extra": extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
