"""One sequence-parallel shard's document-masked attention, sequenced over libhsap.

This is call sequencing and buffer allocation only, one entry point at a
time (the library's hsap_executor runs the same sequence natively, one call
per stage); every step of the path runs inside the library:

  plan      hsap_plan (host C++) -> hsap_split_length / hsap_plan_runs ->
            upload of the lists, hsap_doc_start (device)
  forward   hsap_partial_attn_fwd over the runs (one launch for every chunk,
            or one launch per ring step), then hsap_lse_merge of every slot
            the runs wrote; or hsap_attn_fwd_fused, one pass over every chunk
            per q-tile without partials
  backward  hsap_attn_bwd_preprocess, hsap_partial_attn_bwd (dK/dV over the
            k-major runs, dQ over one run per q-tile across every chunk),
            and hsap_convert_f32_bf16 for the gradients

Tensors follow the library's layouts: the shard's q / dO are [n, Hq, d] in
its local row order; k / v and the dK / dV accumulators are in sharded order
[P, n, Hkv, d]; partial outputs are [slots, n, Hq, d] fp32 with LSE
[slots, Hq, n], where slot = chunk + P * piece (piece > 0 only for split runs).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np
import torch

from . import _lib as L

def _resident_workgroups(device, desc) -> int:
    """Forward workgroups resident on ``device`` for the shapes in ``desc``: the HIP runtime's
    occupancy of the partial-forward kernel the library dispatches, times the compute units
    (hsap_fwd_resident_workgroups)."""
    with torch.cuda.device(device):
        return L.fwd_resident_workgroups(desc)


class ShardAttention:
    """Plan and run one shard of packed, document-masked causal attention.

    ``max_run_tiles``: longest q-major run before it is split into pieces
    (split-K over partial slots); None picks it from the plan and the number
    of resident workgroups (hsap_split_length), 0 disables splitting.
    """

    def __init__(self, cu_seqlens, total_tokens: int, sp_degree: int, layout, shard_id: int, heads_q: int,
                 heads_kv: int, head_dim: int, block_m: int = 128, block_n: int = 128,
                 softmax_scale: Optional[float] = None, device: str = "cuda", max_run_tiles: Optional[int] = None):
        self.device = torch.device(device)
        self.cu_host = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.N = int(total_tokens)
        self.P = int(sp_degree)
        self.n = self.N // self.P
        self.hq, self.hkv, self.d = int(heads_q), int(heads_kv), int(head_dim)
        self.scale = float(softmax_scale) if softmax_scale is not None else 1.0 / math.sqrt(head_dim)
        self.shard = L.shard_desc(total_tokens, sp_degree, layout, shard_id, block_m, block_n)
        self.desc = L.attn_desc(self.shard, heads_q, heads_kv, head_dim, self.scale)
        self.max_run_tiles = max_run_tiles
        self.planned = False

    def _split(self, num_tiles: int) -> int:
        if self.max_run_tiles is not None:
            return int(self.max_run_tiles)
        return L.split_length(self.shard, num_tiles, self.hq, _resident_workgroups(self.device, self.desc))

    # ------------------------------------------------------------------ plan
    def plan(self, backward: bool = False) -> Dict:
        """Host planner, run grouping, upload of the lists and doc starts."""
        p = L.plan(self.cu_host, self.shard)
        self.tiles = p["tiles"]
        self.step_offsets = p["step_offsets"]
        self.useful_pairs = p["useful_pairs"]
        self.chunks = [(self.shard.shard_id - s) % self.P for s in range(self.P)]
        self.split = self._split(len(self.tiles))
        tiles_q, runs_q, self.num_slots = L.plan_runs(self.shard, self.tiles, L.MAJOR_Q, self.split)
        self.runs_q_host = runs_q
        self.present = sorted(set(runs_q[:, 0].tolist()))
        dev = self.device
        self.tiles_q = torch.from_numpy(tiles_q.reshape(-1)).to(dev)
        self.runs_q = torch.from_numpy(runs_q.reshape(-1)).to(dev)
        # per ring step run lists, for executing chunk by chunk
        self.runs_q_step = []
        for c in self.chunks:
            sel = runs_q[runs_q[:, 0] % self.P == c]
            self.runs_q_step.append(torch.from_numpy(np.ascontiguousarray(sel).reshape(-1)).to(dev) if len(sel) else None)
        tiles_a, runs_a, _ = L.plan_runs(self.shard, self.tiles, L.MAJOR_Q_ALL)
        self.tiles_all = torch.from_numpy(tiles_a.reshape(-1)).to(dev)
        self.runs_all = torch.from_numpy(runs_a.reshape(-1)).to(dev)
        if backward:
            tiles_k, runs_k, _ = L.plan_runs(self.shard, self.tiles, L.MAJOR_K)
            self.tiles_k = torch.from_numpy(tiles_k.reshape(-1)).to(dev)
            self.runs_k = torch.from_numpy(runs_k.reshape(-1)).to(dev)
        self.cu_dev = torch.from_numpy(self.cu_host).to(dev)
        self.doc_start = torch.empty(self.N, dtype=torch.int32, device=dev)
        L.doc_start(self.cu_dev, self.N, self.doc_start)
        self.planned = True
        return p

    @property
    def total_useful_pairs(self) -> int:
        return int(self.useful_pairs.sum())

    @property
    def chunks_present(self) -> List[int]:
        return sorted(set(s % self.P for s in self.present))

    # ---------------------------------------------------------- allocation
    def alloc_forward(self) -> Dict[str, torch.Tensor]:
        dev = self.device
        return {
            "o_part": torch.empty(self.num_slots, self.n, self.hq, self.d, dtype=torch.float32, device=dev),
            "lse_part": torch.empty(self.num_slots, self.hq, self.n, dtype=torch.float32, device=dev),
            "o": torch.empty(self.n, self.hq, self.d, dtype=torch.bfloat16, device=dev),
            "lse": torch.empty(self.hq, self.n, dtype=torch.float32, device=dev),
        }

    def alloc_backward(self) -> Dict[str, torch.Tensor]:
        dev = self.device
        return {
            "delta": torch.empty(self.hq, self.n, dtype=torch.float32, device=dev),
            "dq_acc": torch.zeros(self.n, self.hq, self.d, dtype=torch.float32, device=dev),
            "dk_acc": torch.zeros(self.P, self.n, self.hkv, self.d, dtype=torch.float32, device=dev),
            "dv_acc": torch.zeros(self.P, self.n, self.hkv, self.d, dtype=torch.float32, device=dev),
            "dq": torch.empty(self.n, self.hq, self.d, dtype=torch.bfloat16, device=dev),
            "dk": torch.empty(self.P, self.n, self.hkv, self.d, dtype=torch.bfloat16, device=dev),
            "dv": torch.empty(self.P, self.n, self.hkv, self.d, dtype=torch.bfloat16, device=dev),
        }

    # -------------------------------------------------------------- forward
    def forward(self, q, k, v, bufs: Dict[str, torch.Tensor], ring_steps: bool = False) -> None:
        """Partial attention against every chunk with tiles, then the merge.

        ``ring_steps=False`` issues one launch covering every chunk;
        ``ring_steps=True`` issues one launch per ring step in ring order (the
        order a ring rank receives chunks).  Both compute the same runs.
        """
        if not self.planned:
            raise RuntimeError("call plan() first")
        if not self.present:
            raise RuntimeError("shard has no tiles")
        if ring_steps:
            for runs in self.runs_q_step:
                if runs is not None:
                    L.partial_attn_fwd_runs(self.desc, q, k, v, self.doc_start, self.tiles_q, runs, bufs["o_part"],
                                       bufs["lse_part"])
        else:
            L.partial_attn_fwd_runs(self.desc, q, k, v, self.doc_start, self.tiles_q, self.runs_q, bufs["o_part"],
                               bufs["lse_part"])
        L.lse_merge([bufs["o_part"][s] for s in self.present], [bufs["lse_part"][s] for s in self.present],
                    self.n, self.hq, self.d, bufs["o"], bufs["lse"])

    def forward_fused(self, q, k, v, bufs: Dict[str, torch.Tensor]) -> None:
        """The fused forward: final O and LSE into bufs["o"], bufs["lse"], no partials."""
        if not self.planned:
            raise RuntimeError("call plan() first")
        L.attn_fwd_fused(self.desc, q, k, v, self.doc_start, self.tiles_all, self.runs_all, bufs["o"], bufs["lse"])

    # ------------------------------------------------------------- backward
    def backward(self, q, k, v, d_o, fwd: Dict[str, torch.Tensor], bufs: Dict[str, torch.Tensor],
                 zero: bool = True) -> None:
        """dQ for the shard and dK/dV contributions to every chunk, as bf16."""
        if not hasattr(self, "runs_k"):
            raise RuntimeError("call plan(backward=True) first")
        present = self.chunks_present
        if zero:
            bufs["dq_acc"].zero_()
            for c in present:
                bufs["dk_acc"][c].zero_()
                bufs["dv_acc"][c].zero_()
        L.attn_bwd_preprocess(fwd["o"], d_o, self.n, self.hq, self.d, bufs["delta"])
        # dQ over the one-run-per-q-tile lists (every chunk), so each q-tile has one owner
        L.partial_attn_bwd_runs(self.desc, q, k, v, d_o, fwd["lse"], bufs["delta"], self.doc_start, self.tiles_k,
                           self.runs_k, self.tiles_all, self.runs_all, bufs["dq_acc"], bufs["dk_acc"], bufs["dv_acc"])
        L.convert_f32_bf16(bufs["dq_acc"], bufs["dq"])
        # only chunks with tiles receive gradient; the others are zero
        for c in range(self.P):
            if c in present:
                L.convert_f32_bf16(bufs["dk_acc"][c], bufs["dk"][c])
                L.convert_f32_bf16(bufs["dv_acc"][c], bufs["dv"][c])
            elif zero:
                bufs["dk_acc"][c].zero_()
                bufs["dv_acc"][c].zero_()
                bufs["dk"][c].zero_()
                bufs["dv"][c].zero_()


def to_sharded(shard: L.ShardDesc, x: torch.Tensor) -> torch.Tensor:
    """Global-order device tensor [N, ...] -> sharded order [P, n, ...] (hsap_shard_gather)."""
    out = torch.empty_like(x)
    L.shard_gather(shard, x, out)
    P = shard.sp_degree
    return out.view(P, x.shape[0] // P, *x.shape[1:])
