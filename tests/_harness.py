"""Shared helpers of the parity tests: run one shard on the GPU through the C ABI
and the same shard through the fp64 oracle, on the same seeded inputs."""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

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

    # --------------------------------------------------------------- oracle
    def run_oracle(self, rows=None) -> Dict:
        q, k, v = self.q.float().numpy(), self.k.float().numpy(), self.v.float().numpy()
        if self.backward:
            return oracle.shard_backward(q, k, v, self.do.float().numpy(), self.cu, self.N, self.P, self.layout,
                                         self.shard)
        return oracle.shard_forward(q, k, v, self.cu, self.N, self.P, self.layout, self.shard, rows=rows)


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


def rel_max(a, b) -> float:
    den = float(np.max(np.abs(b)))
    return max_abs(a, b) / den if den > 0 else max_abs(a, b)


def compare_backward(gpu: Dict, ref: Dict) -> Dict[str, float]:
    report = {"dq": rel_max(gpu["dq"], ref["dq"]), "dk": rel_max(gpu["dk"], ref["dk"]),
              "dv": rel_max(gpu["dv"], ref["dv"])}
    for key in ("dq", "dk", "dv"):
        assert report[key] <= GRAD_RTOL, report
    return report
