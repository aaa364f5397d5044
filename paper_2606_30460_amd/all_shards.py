"""Every shard of one packed sequence on one GPU: the ranks of a sequence-parallel
group simulated one after another, each running the rank blocks its schedule
gives it.

A rank block (r, c) is shard r's queries against chunk c (compile step 1 of
the SAP section, hsap_load_matrix sizes them).  Two schedules:

  ring      block (r, c) runs on rank r once chunk c's K/V reach it;
  balanced  hsap_balance moves some blocks (r, c) to rank c, the owner of
            chunk c, which receives Q_r instead and sends the partial O and
            LSE back (compile step 2's workload balancing, with the transfer
            of Q blocks of the memory and communication section).

Either way every block is computed by the same runs of shard r's plan into
shard r's partial slots, and rank r merges its own partials, so both
schedules give the same bits.  What differs is how the work falls on the
ranks: each rank's blocks run back to back, timed with HIP events, and the
slowest rank sets the critical path of the step.  No data moves between
ranks here (one GPU holds every chunk); the bytes a real group would move are
counted from the schedule.

This module sequences library calls only: the plan, the balance, the partial
attention and the merge all run inside libhsap.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np
import torch

from . import _lib as L
from .shard_attention import _resident_workgroups


class AllShards:
    """Plan and run all P shards of one packed sequence under the ring or the balanced schedule.

    ``max_run_tiles``: split length of each shard's q-major runs (None: hsap_split_length
    for that shard, as a one-shard run picks it; 0: no split).
    """

    def __init__(self, cu_seqlens, total_tokens: int, sp_degree: int, layout, heads_q: int, heads_kv: int,
                 head_dim: int, block_m: int = 128, block_n: int = 128, softmax_scale: Optional[float] = None,
                 balance: bool = False, max_run_tiles: Optional[int] = None, device: str = "cuda"):
        self.device = torch.device(device)
        self.cu_host = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.N, self.P = int(total_tokens), int(sp_degree)
        self.n = self.N // self.P
        self.layout = layout
        self.hq, self.hkv, self.d = int(heads_q), int(heads_kv), int(head_dim)
        self.bm, self.bn = int(block_m), int(block_n)
        self.scale = float(softmax_scale) if softmax_scale is not None else 1.0 / math.sqrt(head_dim)
        self.balance = bool(balance)
        self.max_run_tiles = max_run_tiles
        self.planned = False

    # ------------------------------------------------------------------ plan
    def plan(self, backward: bool = False) -> None:
        P, dev = self.P, self.device
        base = L.shard_desc(self.N, P, self.layout, 0, self.bm, self.bn)
        self.block_tiles, self.block_pairs = L.load_matrix(self.cu_host, base)
        if self.balance:
            self.exec_rank, self.rank_tiles = L.balance(self.block_tiles)
        else:
            self.exec_rank = np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
            self.rank_tiles = self.block_tiles.sum(axis=1)
        self.cu_dev = torch.from_numpy(self.cu_host).to(dev)
        self.doc_start = torch.empty(self.N, dtype=torch.int32, device=dev)
        L.doc_start(self.cu_dev, self.N, self.doc_start)
        resident = _resident_workgroups(dev, L.attn_desc(base, self.hq, self.hkv, self.d, self.scale))
        self.descs, self.tiles_dev, self.parts = [], [], []
        # runs[e][r]: device run list of shard r's blocks that rank e computes (None if none)
        self.runs: List[List[Optional[torch.Tensor]]] = [[None] * P for _ in range(P)]
        for r in range(P):
            shard = L.shard_desc(self.N, P, self.layout, r, self.bm, self.bn)
            self.descs.append(L.attn_desc(shard, self.hq, self.hkv, self.d, self.scale))
            tiles = L.plan(self.cu_host, shard)["tiles"]
            split = self.max_run_tiles
            if split is None:
                split = L.split_length(shard, len(tiles), self.hq, resident)
            sorted_tiles, runs, _ = L.plan_runs(shard, tiles, L.MAJOR_Q, split)
            # partial slots renumbered densely, in increasing slot order (the merge order)
            present = sorted(set(runs[:, 0].tolist()))
            dense = {s: i for i, s in enumerate(present)}
            runs = runs.copy()
            chunk_of_run = runs[:, 0] % P
            runs[:, 0] = [dense[s] for s in runs[:, 0].tolist()]
            self.parts.append(len(present))
            self.tiles_dev.append(torch.from_numpy(np.ascontiguousarray(sorted_tiles).reshape(-1)).to(dev))
            for e in range(P):
                sel = runs[self.exec_rank[r, chunk_of_run] == e]
                if len(sel):
                    self.runs[e][r] = torch.from_numpy(np.ascontiguousarray(sel).reshape(-1)).to(dev)
        self.backward_planned = False
        if backward:
            self._plan_backward()
        self.planned = True

    def _plan_backward(self) -> None:
        """Per block (r, c): shard r's unsplit q-major runs of chunk c (dQ kernel) and its k-major runs
        of chunk c (dK/dV kernel); the part indices of every shard's dQ and every chunk's dK/dV."""
        P, dev = self.P, self.device
        self.dq_parts = [[c for c in range(P) if self.block_tiles[r, c] > 0] for r in range(P)]
        self.dkv_parts = [[r for r in range(P) if self.block_tiles[r, c] > 0] for c in range(P)]
        self.bwd_tiles_q, self.bwd_tiles_k = [], []
        self.bwd_runs: Dict[tuple, tuple] = {}
        for r in range(P):
            shard = self.descs[r].shard
            tiles = L.plan(self.cu_host, shard)["tiles"]
            sq, rq, _ = L.plan_runs(shard, tiles, L.MAJOR_Q, 0)     # unsplit: slot = chunk
            sk, rk, _ = L.plan_runs(shard, tiles, L.MAJOR_K, 0)     # slot = chunk
            self.bwd_tiles_q.append(torch.from_numpy(np.ascontiguousarray(sq).reshape(-1)).to(dev))
            self.bwd_tiles_k.append(torch.from_numpy(np.ascontiguousarray(sk).reshape(-1)).to(dev))
            for c in self.dq_parts[r]:
                self.bwd_runs[(r, c)] = tuple(torch.from_numpy(np.ascontiguousarray(x[x[:, 0] == c]).reshape(-1)).to(dev)
                                              for x in (rq, rk))
        self.backward_planned = True

    # ------------------------------------------------------------ schedule
    def schedule(self) -> Dict:
        """What each rank computes and the bytes a real group would move (per head group)."""
        P, n = self.P, self.n
        kv_bytes = 2 * n * self.hkv * self.d * 2            # one chunk's K and V, bf16
        q_bytes = n * self.hq * self.d * 2                  # one shard's Q, bf16
        o_bytes = n * self.hq * (self.d + 1) * 4            # one partial O and LSE back, fp32
        kv_moved = q_moved = 0
        for r in range(P):
            for c in range(P):
                if r == c or self.block_tiles[r, c] == 0:
                    continue
                if self.exec_rank[r, c] == r:
                    kv_moved += kv_bytes
                else:
                    q_moved += q_bytes + o_bytes
        rank_pairs = np.zeros(P, dtype=np.int64)
        for r in range(P):
            for c in range(P):
                rank_pairs[self.exec_rank[r, c]] += self.block_pairs[r, c]
        mean = float(self.rank_tiles.mean())
        return {"rank_tiles": self.rank_tiles.tolist(), "rank_pairs": rank_pairs.tolist(),
                "tile_imbalance": float(self.rank_tiles.max()) / mean if mean > 0 else 1.0,
                "moved_blocks": int(sum(1 for r in range(P) for c in range(P)
                                        if r != c and self.block_tiles[r, c] and self.exec_rank[r, c] == c)),
                "kv_bytes_moved": int(kv_moved), "q_o_bytes_moved": int(q_moved)}

    # ------------------------------------------------------------ execution
    def alloc(self) -> Dict[str, object]:
        dev = self.device
        return {
            "o_part": [torch.empty(p, self.n, self.hq, self.d, dtype=torch.float32, device=dev) for p in self.parts],
            "lse_part": [torch.empty(p, self.hq, self.n, dtype=torch.float32, device=dev) for p in self.parts],
            "o": torch.empty(self.P, self.n, self.hq, self.d, dtype=torch.bfloat16, device=dev),
            "lse": torch.empty(self.P, self.hq, self.n, dtype=torch.float32, device=dev),
        }

    def forward(self, q, k, v, bufs: Dict[str, object], timed: bool = False) -> Optional[Dict[str, List[float]]]:
        """q [P, n, Hq, d] (every shard, sharded order), k / v [P, n, Hkv, d] -> bufs["o"] [P, n, Hq, d],
        bufs["lse"] [P, Hq, n].  Rank e runs its blocks, then merges shard e; with ``timed`` the
        milliseconds of each rank's blocks and of its merge are returned."""
        if not self.planned:
            raise RuntimeError("call plan() first")
        P = self.P
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(P)] if timed else None
        for e in range(P):
            if timed:
                ev[e][0].record()
            for r in range(P):
                runs = self.runs[e][r]
                if runs is not None:
                    L.partial_attn_fwd_runs(self.descs[r], q[r], k, v, self.doc_start, self.tiles_dev[r], runs,
                                       bufs["o_part"][r], bufs["lse_part"][r])
            if timed:
                ev[e][1].record()
        # every partial of a shard exists only once all ranks are done (a block may run on another rank)
        for r in range(P):
            if timed:
                ev[r][2].record()
            parts = self.parts[r]
            L.lse_merge([bufs["o_part"][r][i] for i in range(parts)], [bufs["lse_part"][r][i] for i in range(parts)],
                        self.n, self.hq, self.d, bufs["o"][r], bufs["lse"][r])
            if timed:
                ev[r][3].record()
        if not timed:
            return None
        torch.cuda.synchronize()
        return {"blocks_ms": [ev[e][0].elapsed_time(ev[e][1]) for e in range(P)],
                "merge_ms": [ev[r][2].elapsed_time(ev[r][3]) for r in range(P)]}

    # ------------------------------------------------------------ backward
    def alloc_backward(self) -> Dict[str, object]:
        dev, n, f32 = self.device, self.n, torch.float32
        return {
            "delta": torch.empty(self.P, self.hq, n, dtype=f32, device=dev),
            "dq_part": [torch.empty(max(len(x), 1), n, self.hq, self.d, dtype=f32, device=dev) for x in self.dq_parts],
            "dk_part": [torch.empty(max(len(x), 1), n, self.hkv, self.d, dtype=f32, device=dev) for x in self.dkv_parts],
            "dv_part": [torch.empty(max(len(x), 1), n, self.hkv, self.d, dtype=f32, device=dev) for x in self.dkv_parts],
            "dq": torch.empty(self.P, n, self.hq, self.d, dtype=torch.bfloat16, device=dev),
            "dk": torch.empty(self.P, n, self.hkv, self.d, dtype=torch.bfloat16, device=dev),
            "dv": torch.empty(self.P, n, self.hkv, self.d, dtype=torch.bfloat16, device=dev),
        }

    def backward(self, q, k, v, d_o, o, lse, bufs: Dict[str, object],
                 timed: bool = False) -> Optional[Dict[str, List[float]]]:
        """Gradients of every shard's attention: q, d_o, o [P, n, Hq, d], lse [P, Hq, n] (the forward's
        outputs), k / v [P, n, Hkv, d] -> bufs["dq"] [P, n, Hq, d], bufs["dk"] / bufs["dv"] [P, n, Hkv, d]
        (bf16; chunks without any block are left as they are).  Rank e differentiates the blocks
        its schedule gives it, each into its own zeroed fp32 parts (hsap_partial_attn_bwd); then
        every shard's dQ parts and every chunk's dK/dV parts are summed in part order
        (hsap_sum_parts), so any schedule gives the same bits.  With ``timed`` the milliseconds of
        each rank's blocks and of its sums are returned."""
        if not (self.planned and self.backward_planned):
            raise RuntimeError("call plan(backward=True) first")
        P = self.P
        for r in range(P):
            L.attn_bwd_preprocess(o[r], d_o[r], self.n, self.hq, self.d, bufs["delta"][r])
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(P)] if timed else None
        for e in range(P):
            if timed:
                ev[e][0].record()
            for r in range(P):
                for c in self.dq_parts[r]:
                    if self.exec_rank[r, c] != e:
                        continue
                    dq_t = bufs["dq_part"][r][self.dq_parts[r].index(c)]
                    i = self.dkv_parts[c].index(r)
                    dk_t, dv_t = bufs["dk_part"][c][i], bufs["dv_part"][c][i]
                    for t_ in (dq_t, dk_t, dv_t):
                        t_.zero_()
                    runs_q, runs_k = self.bwd_runs[(r, c)]
                    L.partial_attn_bwd_runs(self.descs[r], q[r], k[c], v[c], d_o[r], lse[r], bufs["delta"][r],
                                       self.doc_start, self.bwd_tiles_k[r], runs_k, self.bwd_tiles_q[r], runs_q,
                                       dq_t, dk_t, dv_t, kv_chunk=c)
            if timed:
                ev[e][1].record()
        for x in range(P):
            if timed:
                ev[x][2].record()
            if self.dq_parts[x]:
                L.sum_parts([bufs["dq_part"][x][i] for i in range(len(self.dq_parts[x]))], bufs["dq"][x])
            if self.dkv_parts[x]:
                L.sum_parts([bufs["dk_part"][x][i] for i in range(len(self.dkv_parts[x]))], bufs["dk"][x])
                L.sum_parts([bufs["dv_part"][x][i] for i in range(len(self.dkv_parts[x]))], bufs["dv"][x])
            if timed:
                ev[x][3].record()
        if not timed:
            return None
        torch.cuda.synchronize()
        return {"blocks_ms": [ev[e][0].elapsed_time(ev[e][1]) for e in range(P)],
                "sum_ms": [ev[x][2].elapsed_time(ev[x][3]) for x in range(P)]}
