"""Shared helpers of the parity tests: run one shard on the GPU through the C ABI
and the same shard through the fp64 oracle, on the same seeded inputs."""
from __future__ import annotations

import concurrent.futures
import os
from typing import Dict, Optional

import numpy as np
import torch
from threadpoolctl import threadpool_limits

import oracle
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.shard_attention import ShardAttention, to_sharded

# tolerances the comparison must meet (bf16 inputs, fp32 accumulation)
O_ATOL = 2e-2        # final and partial O, max-abs
LSE_ATOL = 1e-3      # natural-log units, max-abs
GRAD_RTOL = 3e-2     # max|g - g_ref| / max|g_ref|, per gradient


def critical_shard(cu, N, P, layout, bm, bn) -> int:
    """Shard with the most allowed pairs (ties: lowest id), from the library planner."""
    best, best_r = -1, 0
    for r in range(P):
        pairs = int(L.plan(cu, L.shard_desc(N, P, layout, r, bm, bn))["useful_pairs"].sum())
        if pairs > best:
            best, best_r = pairs, r
    return best_r


class Case:
    """Inputs of one problem, on the CPU (bf16) and on the GPU (sharded order)."""

    def __init__(self, cu, N, P, layout, shard, hq, hkv, d, bm, bn, seed=0, backward=False, q_zero=False):
        self.cu = np.asarray(cu, dtype=np.int32)
        self.N, self.P, self.layout, self.shard = N, P, layout, shard
        self.hq, self.hkv, self.d, self.bm, self.bn = hq, hkv, d, bm, bn
        from workloads import random_bf16
        self.q = random_bf16((N, hq, d), seed + 1)
        if q_zero:
            self.q.zero_()
        self.k = random_bf16((N, hkv, d), seed + 2)
        self.v = random_bf16((N, hkv, d), seed + 3)
        self.do = random_bf16((N, hq, d), seed + 4) if backward else None
        self.backward = backward

    @classmethod
    def from_workload(cls, w, shard: Optional[int] = None):
        r = w.shard if shard is None else shard
        if r is None:
            r = critical_shard(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, w.block_m, w.block_n)
        return cls(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, r, w.heads_q, w.heads_kv, w.head_dim,
                   w.block_m, w.block_n, w.seed, w.backward)

    # ------------------------------------------------------------------ GPU
    def run_gpu(self, ring_steps: bool = False, max_run_tiles=None) -> Dict[str, np.ndarray]:
        sa = ShardAttention(self.cu, self.N, self.P, self.layout, self.shard, self.hq, self.hkv, self.d,
                            self.bm, self.bn, max_run_tiles=max_run_tiles)
        sa.plan(backward=self.backward)
        dev = torch.device("cuda")
        q_sh = to_sharded(sa.shard, self.q.to(dev))[self.shard].contiguous()
        k_sh = to_sharded(sa.shard, self.k.to(dev))
        v_sh = to_sharded(sa.shard, self.v.to(dev))
        fwd = sa.alloc_forward()
        fwd["lse_part"].fill_(float("nan"))       # rows never written stay NaN and fail the comparison
        sa.forward(q_sh, k_sh, v_sh, fwd, ring_steps=ring_steps)
        out = {"sa": sa, "o": fwd["o"].float().cpu().numpy(), "lse": fwd["lse"].cpu().numpy(),
               "o_part": fwd["o_part"].cpu().numpy(), "lse_part": fwd["lse_part"].cpu().numpy()}
        fused = {"o": torch.full_like(fwd["o"], float("nan")), "lse": torch.full_like(fwd["lse"], float("nan"))}
        sa.forward_fused(q_sh, k_sh, v_sh, fused)
        out["o_fused"] = fused["o"].float().cpu().numpy()
        out["lse_fused"] = fused["lse"].cpu().numpy()
        if self.backward:
            do_sh = to_sharded(sa.shard, self.do.to(dev))[self.shard].contiguous()
            bwd = sa.alloc_backward()
            sa.backward(q_sh, k_sh, v_sh, do_sh, fwd, bwd)
            out.update({"dq": bwd["dq_acc"].cpu().numpy(), "dk": bwd["dk_acc"].cpu().numpy(),
                        "dv": bwd["dv_acc"].cpu().numpy(), "delta": bwd["delta"].cpu().numpy(),
                        "dq_bf16": bwd["dq"].float().cpu().numpy()})
        torch.cuda.synchronize()
        return out

    def run_executor(self, max_run_tiles: int = -1, cu=None) -> Dict[str, np.ndarray]:
        """The same shard through one hsap_executor: plan, forward (partial + merge, and
        fused), backward when the case has one.  ``cu`` plans other documents on the
        same inputs."""
        s = L.shard_desc(self.N, self.P, self.layout, self.shard, self.bm, self.bn)
        desc = L.attn_desc(s, self.hq, self.hkv, self.d, 1.0 / float(np.sqrt(self.d)))
        ex = L.Executor(desc, backward=self.backward, fused=True, max_run_tiles=max_run_tiles)
        try:
            dev = torch.device("cuda")
            q_sh = to_sharded(s, self.q.to(dev))[self.shard].contiguous()
            k_sh = to_sharded(s, self.k.to(dev))
            v_sh = to_sharded(s, self.v.to(dev))
            ex.plan(self.cu if cu is None else cu)
            n = self.N // self.P
            o = torch.full((n, self.hq, self.d), float("nan"), dtype=torch.bfloat16, device=dev)
            lse = torch.full((self.hq, n), float("nan"), dtype=torch.float32, device=dev)
            ex.forward(q_sh, k_sh, v_sh, o, lse)
            of, lsef = torch.full_like(o, float("nan")), torch.full_like(lse, float("nan"))
            ex.forward(q_sh, k_sh, v_sh, of, lsef, fused=True)
            os_, lses = torch.full_like(o, float("nan")), torch.full_like(lse, float("nan"))
            ex.partial_forward(q_sh, k_sh, v_sh, os_, lses)     # the same forward as two stage calls
            ex.merge(os_, lses)
            out = {"info": ex.info(), "o": o.float().cpu().numpy(), "lse": lse.cpu().numpy(),
                   "o_fused": of.float().cpu().numpy(), "lse_fused": lsef.cpu().numpy(),
                   "o_staged": os_.float().cpu().numpy(), "lse_staged": lses.cpu().numpy()}
            if self.backward:
                do_sh = to_sharded(s, self.do.to(dev))[self.shard].contiguous()
                # chunks without tiles are not written: the caller's zeros stay (their gradient is zero)
                dq = torch.full_like(q_sh, float("nan"))
                dk, dv = torch.zeros_like(k_sh), torch.zeros_like(v_sh)
                mask = ex.info()["chunk_mask"]
                for chunk in range(self.P):
                    if mask >> chunk & 1:
                        dk[chunk].fill_(float("nan"))
                        dv[chunk].fill_(float("nan"))
                ex.backward(q_sh, k_sh, v_sh, do_sh, o, lse, dq, dk, dv)
                out.update({"dq": dq.float().cpu().numpy(), "dk": dk.float().cpu().numpy(),
                            "dv": dv.float().cpu().numpy()})
            torch.cuda.synchronize()
            return out
        finally:
            ex.close()

    def run_tile_list(self, backward: Optional[bool] = None) -> Dict[str, np.ndarray]:
        """The shard through the boundary's tile-list calls, ring step by ring step: hsap_plan, then
        per chunk c hsap_partial_attn_fwd on the step's tiles (one chunk's K/V passed alone) into
        its own partial, hsap_lse_merge of the partials of the chunks with tiles; with the backward,
        hsap_attn_bwd_preprocess and per chunk hsap_partial_attn_bwd accumulating dQ and that
        chunk's dK/dV.  Partials and gradients are pre-filled with NaN / zero."""
        bwd = self.backward if backward is None else backward
        s = L.shard_desc(self.N, self.P, self.layout, self.shard, self.bm, self.bn)
        dev = torch.device("cuda")
        p = L.plan(self.cu, s)
        offs = p["step_offsets"]
        n = self.N // self.P
        q = to_sharded(s, self.q.to(dev))[self.shard].contiguous()
        k, v = to_sharded(s, self.k.to(dev)), to_sharded(s, self.v.to(dev))
        doc_start = torch.empty(self.N, dtype=torch.int32, device=dev)
        L.doc_start(torch.from_numpy(self.cu).to(dev), self.N, doc_start)
        o_part = torch.full((self.P, n, self.hq, self.d), float("nan"), dtype=torch.float32, device=dev)
        lse_part = torch.full((self.P, self.hq, n), float("nan"), dtype=torch.float32, device=dev)
        chunks, lists = [], {}
        for step in range(self.P):
            c = (self.shard - step) % self.P
            chunks.append(c)
            lists[c] = torch.from_numpy(np.ascontiguousarray(p["tiles"][offs[step]:offs[step + 1]]).reshape(-1)).to(dev)
            desc = L.attn_desc(s, self.hq, self.hkv, self.d, 1.0 / float(np.sqrt(self.d)), chunk_id=c)
            L.partial_attn_fwd(desc, q, k[c], v[c], doc_start, lists[c], o_part[c], lse_part[c])
        present = [c for c in sorted(chunks) if lists[c].numel()]
        o = torch.empty(n, self.hq, self.d, dtype=torch.bfloat16, device=dev)
        lse = torch.empty(self.hq, n, dtype=torch.float32, device=dev)
        L.lse_merge([o_part[c] for c in present], [lse_part[c] for c in present], n, self.hq, self.d, o, lse)
        out = {"chunks": chunks, "o_part": o_part.cpu().numpy(), "lse_part": lse_part.cpu().numpy(),
               "o": o.float().cpu().numpy(), "lse": lse.cpu().numpy(), "tiles": p["tiles"], "step_offsets": offs}
        if bwd:
            d_o = to_sharded(s, self.do.to(dev))[self.shard].contiguous()
            delta = torch.empty(self.hq, n, dtype=torch.float32, device=dev)
            L.attn_bwd_preprocess(o, d_o, n, self.hq, self.d, delta)
            dq = torch.zeros(n, self.hq, self.d, dtype=torch.float32, device=dev)
            dk = torch.zeros(self.P, n, self.hkv, self.d, dtype=torch.float32, device=dev)
            dv = torch.zeros_like(dk)
            for c in chunks:        # ring order: dQ accumulates over the chunks, dK/dV per chunk
                desc = L.attn_desc(s, self.hq, self.hkv, self.d, 1.0 / float(np.sqrt(self.d)), chunk_id=c)
                L.partial_attn_bwd(desc, q, k[c], v[c], d_o, lse, delta, doc_start, lists[c], dq, dk[c], dv[c])
            out.update(dq=dq.cpu().numpy(), dk=dk.cpu().numpy(), dv=dv.cpu().numpy())
        torch.cuda.synchronize()
        return out

    # --------------------------------------------------------------- oracle
    def run_oracle(self, rows=None, kv_heads=None, backward=None) -> Dict:
        """The fp64 oracle on this case (backward when the case has one, unless ``backward`` says
        otherwise).  Heads are independent problems, so the work is split by K/V head over host
        threads (each oracle call sees a plain head subset) and the results are put back together
        along the head axes; ``kv_heads`` restricts it to those K/V heads and their query heads."""
        bwd = self.backward if backward is None else backward
        kv = list(range(self.hkv)) if kv_heads is None else [int(g) for g in kv_heads]
        q, k, v = self.q.float().numpy(), self.k.float().numpy(), self.v.float().numpy()
        do = self.do.float().numpy() if bwd else None
        return oracle_by_kv_heads(q, k, v, do, self.cu, self.N, self.P, self.layout, self.shard, kv, rows=rows)

    def q_heads(self, kv_heads) -> np.ndarray:
        """Query heads that read the given K/V heads, in order."""
        group = self.hq // self.hkv
        return np.concatenate([np.arange(g * group, (g + 1) * group) for g in kv_heads])


def _oracle_workers() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def oracle_by_kv_heads(q, k, v, do, cu, N, P, layout, shard, kv_heads, rows=None) -> Dict:
    """oracle.shard_forward (do is None) or oracle.shard_backward for the given K/V heads and the
    query heads that read them, one K/V head per task on a pool of host threads, each calling a
    single-threaded BLAS; results are concatenated along the head axes in the order of ``kv_heads``.

    The BLAS runs single-threaded because its own thread pool is shared by every caller thread:
    OpenBLAS documents that a program which is itself multi-threaded must set it to one thread,
    since concurrent calls into its threaded kernels conflict."""
    hq, hkv = q.shape[1], k.shape[1]
    group = hq // hkv

    def one(g):
        hs = slice(g * group, (g + 1) * group)
        if do is None:
            return oracle.shard_forward(q[:, hs], k[:, g:g + 1], v[:, g:g + 1], cu, N, P, layout, shard, rows=rows)
        if rows is not None:
            raise ValueError("the backward is computed over every row")
        return oracle.shard_backward(q[:, hs], k[:, g:g + 1], v[:, g:g + 1], do[:, hs], cu, N, P, layout, shard)

    with threadpool_limits(limits=1):
        with concurrent.futures.ThreadPoolExecutor(min(_oracle_workers(), len(kv_heads))) as pool:
            parts = list(pool.map(one, kv_heads))

    def fwd_cat(fs):
        return {"chunks": fs[0]["chunks"], "q_pos": fs[0]["q_pos"],
                "o_parts": [np.concatenate([f["o_parts"][i] for f in fs], axis=1) for i in range(len(fs[0]["chunks"]))],
                "lse_parts": [np.concatenate([f["lse_parts"][i] for f in fs], axis=0)
                              for i in range(len(fs[0]["chunks"]))],
                "o": np.concatenate([f["o"] for f in fs], axis=1), "lse": np.concatenate([f["lse"] for f in fs], axis=0)}

    if do is None:
        return fwd_cat(parts)
    out = fwd_cat([p["fwd"] for p in parts])
    return {"dq": np.concatenate([p["dq"] for p in parts], axis=1),
            "dk": np.concatenate([p["dk"] for p in parts], axis=2),
            "dv": np.concatenate([p["dv"] for p in parts], axis=2),
            "o": out["o"], "lse": out["lse"], "delta": np.concatenate([p["delta"] for p in parts], axis=0),
            "fwd": out}


def max_abs(a, b) -> float:
    return float(np.max(np.abs(np.asarray(a, dtype=np.float64) - np.asarray(b, dtype=np.float64)))) if np.size(a) else 0.0


def compare_forward(gpu: Dict, ref: Dict, rows=None) -> Dict[str, float]:
    """Partial and merged outputs of the GPU against the oracle (asserts the bars).

    A chunk whose runs were split writes several slots; those pieces are
    combined on the host first, so every chunk is compared with the oracle's
    partial for it."""
    sl = slice(None) if rows is None else np.asarray(rows)
    report = {}
    sa = gpu["sa"]
    assert ref["chunks"] == sa.chunks
    for step, c in enumerate(ref["chunks"]):
        lse_ref = ref["lse_parts"][step]                     # [Hq, rows]
        slots = [s for s in sa.present if s % sa.P == c]
        if not slots:
            assert np.all(np.isneginf(lse_ref)), "oracle finds allowed keys in chunk %d the planner skipped" % c
            continue
        for s in slots:
            assert not np.any(np.isnan(gpu["lse_part"][s][:, sl])), "unwritten LSE rows in slot %d" % s
        if len(slots) == 1:
            lse_g, o_g = gpu["lse_part"][slots[0]][:, sl], gpu["o_part"][slots[0]][sl]
        else:
            o_g, lse_g = oracle.lse_merge([gpu["o_part"][s][sl] for s in slots],
                                          [gpu["lse_part"][s][:, sl] for s in slots])
        ninf_ref, ninf_g = np.isneginf(lse_ref), np.isneginf(lse_g)
        assert np.array_equal(ninf_ref, ninf_g), "-inf rows differ in chunk %d" % c
        fin = ~ninf_ref
        report["lse_part_%d" % c] = max_abs(lse_g[fin], lse_ref[fin])
        assert report["lse_part_%d" % c] <= LSE_ATOL, report
        fin_rows = fin.T                                      # [rows, Hq]
        report["o_part_%d" % c] = max_abs(o_g[fin_rows], ref["o_parts"][step][fin_rows])
        assert report["o_part_%d" % c] <= O_ATOL, report
    report["o"] = max_abs(gpu["o"][sl], ref["o"])
    report["lse"] = max_abs(gpu["lse"][:, sl], ref["lse"])
    assert report["o"] <= O_ATOL, report
    assert report["lse"] <= LSE_ATOL, report
    if "o_fused" in gpu:                                  # the fused forward meets the same bar
        report["o_fused"] = max_abs(gpu["o_fused"][sl], ref["o"])
        report["lse_fused"] = max_abs(gpu["lse_fused"][:, sl], ref["lse"])
        assert report["o_fused"] <= O_ATOL, report
        assert report["lse_fused"] <= LSE_ATOL, report
    return report


def compare_tile_list(gpu: Dict, ref: Dict) -> Dict[str, float]:
    """Per-chunk partials of the tile-list calls and their merge against the oracle (asserts the bars;
    the -inf rows of every chunk's partial must be the oracle's exactly, and none may be NaN)."""
    report = {}
    for step, c in enumerate(ref["chunks"]):
        lse_g, lse_r = gpu["lse_part"][c], ref["lse_parts"][step]
        assert not np.isnan(lse_g).any(), "LSE rows of chunk %d not written" % c
        assert np.array_equal(np.isneginf(lse_g), np.isneginf(lse_r)), "-inf rows differ in chunk %d" % c
        fin = ~np.isneginf(lse_r)
        report["lse_part_%d" % c] = max_abs(lse_g[fin], lse_r[fin])
        report["o_part_%d" % c] = max_abs(gpu["o_part"][c][fin.T], ref["o_parts"][step][fin.T])
        assert report["lse_part_%d" % c] <= LSE_ATOL and report["o_part_%d" % c] <= O_ATOL, report
    report["o"], report["lse"] = max_abs(gpu["o"], ref["o"]), max_abs(gpu["lse"], ref["lse"])
    assert report["o"] <= O_ATOL and report["lse"] <= LSE_ATOL, report
    return report


def rel_max(a, b) -> float:
    den = float(np.max(np.abs(b)))
    return max_abs(a, b) / den if den > 0 else max_abs(a, b)


def compare_backward(gpu: Dict, ref: Dict) -> Dict[str, float]:
    report = {"dq": rel_max(gpu["dq"], ref["dq"]), "dk": rel_max(gpu["dk"], ref["dk"]),
              "dv": rel_max(gpu["dv"], ref["dv"])}
    for key in ("dq", "dk", "dv"):
        assert report[key] <= GRAD_RTOL, report
    return report
