"""The per-rank instruction lists of one packed sequence's forward pass (hsap_emit_forward) and
backward pass (hsap_emit_backward), executed on one GPU with one HIP stream standing in for each
rank.

Every rank gets the buffers the lists name: its own Q shard and K/V chunk (views of the
sharded inputs), two receive slots for Q and for K/V (one shard or one chunk each: the
partial forward is given the address chunk 0 would have, so that it reads the received
chunk's rows from the slot), two result slots for partials it computes for other shards,
and one part slot per chunk with tiles of its own shard.  A
stage runs on every rank's stream after all ranks finished the previous stage (the batched
point-to-point group of a stage); within it a rank's receives are device copies from the
peer's buffer, its computation is hsap_partial_attn_fwd over that block's q-major runs, and
its merge is hsap_lse_merge.  Sends need no action here: the receiving rank's copy reads
the sender's buffer, which the stage order keeps unchanged until then.

The backward program runs each block on the rank that computed its forward: a ring block
(r, c) on rank r with chunk c's K/V received, its dK/dV part sent back to rank c; a transferred
block on rank c with shard r's Q and dO (plus the shard's final LSE and delta) received, its dQ
part sent back to rank r.  A block's parts come from hsap_partial_attn_bwd (fp32, into zeroed
part buffers: the dQ kernel over the block's q-major runs, the dK/dV kernel over its k-major
runs); each rank sums its dQ parts and its dK/dV parts in part order (hsap_sum_parts) into its
bf16 gradients.  Before stage 0 every rank computes delta = rowsum(dO o O) of its own shard
(hsap_attn_bwd_preprocess): the row term that travels with dO.

This sequences library calls and device copies only; all arithmetic runs in libhsap.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np
import torch

from . import _lib as L


class SapProgram:
    """Emit and run the forward program of all P ranks (ring or balanced assignment)."""

    def __init__(self, cu_seqlens, total_tokens: int, sp_degree: int, layout, heads_q: int, heads_kv: int,
                 head_dim: int, block_m: int = 128, block_n: int = 128, softmax_scale: Optional[float] = None,
                 balance: bool = False, device: str = "cuda"):
        self.device = torch.device(device)
        self.cu_host = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.N, self.P = int(total_tokens), int(sp_degree)
        self.n = self.N // self.P
        self.layout = layout
        self.hq, self.hkv, self.d = int(heads_q), int(heads_kv), int(head_dim)
        self.bm, self.bn = int(block_m), int(block_n)
        self.scale = float(softmax_scale) if softmax_scale is not None else 1.0 / math.sqrt(head_dim)
        self.balance = bool(balance)
        self.planned = False

    def plan(self, backward: bool = False) -> None:
        P, dev = self.P, self.device
        base = L.shard_desc(self.N, P, self.layout, 0, self.bm, self.bn)
        self.block_tiles, _ = L.load_matrix(self.cu_host, base)
        if self.balance:
            self.exec_rank = L.balance(self.block_tiles)[0]
        else:
            self.exec_rank = np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
        self.ops, self.num_stages = L.emit_forward(self.block_tiles, self.exec_rank)
        self.cu_dev = torch.from_numpy(self.cu_host).to(dev)
        self.doc_start = torch.empty(self.N, dtype=torch.int32, device=dev)
        L.doc_start(self.cu_dev, self.N, self.doc_start)
        self.descs, self.tiles_dev, self.runs_host = [], [], []
        for r in range(P):
            shard = L.shard_desc(self.N, P, self.layout, r, self.bm, self.bn)
            self.descs.append(L.attn_desc(shard, self.hq, self.hkv, self.d, self.scale))
            tiles = L.plan(self.cu_host, shard)["tiles"]
            sorted_tiles, runs, _ = L.plan_runs(shard, tiles, L.MAJOR_Q, 0)   # unsplit: slot = chunk
            self.tiles_dev.append(torch.from_numpy(np.ascontiguousarray(sorted_tiles).reshape(-1)).to(dev))
            self.runs_host.append(runs)
        self._runs_dev: Dict[Tuple[int, int, int], torch.Tensor] = {}
        self.parts = [int((self.block_tiles[r] > 0).sum()) for r in range(P)]
        self.backward_planned = False
        if backward:
            self._plan_backward()
        self.planned = True

    def _plan_backward(self) -> None:
        """The backward's instruction lists, part indices and each shard's k-major lists."""
        P, dev = self.P, self.device
        self.ops_bwd, self.num_stages_bwd = L.emit_backward(self.block_tiles, self.exec_rank)
        self.dq_parts = [[c for c in range(P) if self.block_tiles[r, c] > 0] for r in range(P)]
        self.dkv_parts = [[r for r in range(P) if self.block_tiles[r, c] > 0] for c in range(P)]
        self.tiles_k_dev, self.runs_k_host = [], []
        for r in range(P):
            tiles = L.plan(self.cu_host, self.descs[r].shard)["tiles"]
            sorted_k, runs_k, _ = L.plan_runs(self.descs[r].shard, tiles, L.MAJOR_K, 0)    # slot = chunk
            self.tiles_k_dev.append(torch.from_numpy(np.ascontiguousarray(sorted_k).reshape(-1)).to(dev))
            self.runs_k_host.append(runs_k)
        self._runs_k_dev: Dict[Tuple[int, int], torch.Tensor] = {}
        self.backward_planned = True

    def _runs_k(self, r: int, c: int) -> Optional[torch.Tensor]:
        """Block (r, c)'s k-major runs on the device (None when it has none)."""
        key = (r, c)
        if key not in self._runs_k_dev:
            runs = self.runs_k_host[r]
            sel = np.ascontiguousarray(runs[runs[:, 0] == c])
            self._runs_k_dev[key] = torch.from_numpy(sel.reshape(-1)).to(self.device) if len(sel) else None
        return self._runs_k_dev[key]

    def _runs(self, r: int, c: int, slot: int) -> torch.Tensor:
        """Block (r, c)'s runs on the device, writing partial slot ``slot`` of the buffer they get."""
        key = (r, c, slot)
        if key not in self._runs_dev:
            runs = self.runs_host[r]
            sel = np.ascontiguousarray(runs[runs[:, 0] == c])
            sel[:, 0] = slot
            self._runs_dev[key] = torch.from_numpy(sel.reshape(-1)).to(self.device)
        return self._runs_dev[key]

    def alloc(self) -> Dict[str, list]:
        P, n, dev = self.P, self.n, self.device
        bf, f32 = torch.bfloat16, torch.float32
        return {
            "q_recv": [torch.empty(2, n, self.hq, self.d, dtype=bf, device=dev) for _ in range(P)],
            # receive slots hold one chunk each
            "k_recv": [torch.empty(2, n, self.hkv, self.d, dtype=bf, device=dev) for _ in range(P)],
            "v_recv": [torch.empty(2, n, self.hkv, self.d, dtype=bf, device=dev) for _ in range(P)],
            "o_res": [torch.empty(2, n, self.hq, self.d, dtype=f32, device=dev) for _ in range(P)],
            "lse_res": [torch.empty(2, self.hq, n, dtype=f32, device=dev) for _ in range(P)],
            "o_part": [torch.empty(max(p, 1), n, self.hq, self.d, dtype=f32, device=dev) for p in self.parts],
            "lse_part": [torch.empty(max(p, 1), self.hq, n, dtype=f32, device=dev) for p in self.parts],
            "o": torch.empty(P, n, self.hq, self.d, dtype=bf, device=dev),
            "lse": torch.empty(P, self.hq, n, dtype=f32, device=dev),
        }

    def run(self, q, k, v, bufs: Dict[str, list], timed: bool = False) -> Optional[float]:
        """q [P, n, Hq, d], k / v [P, n, Hkv, d] (every rank's own data, sharded order) ->
        bufs["o"] [P, n, Hq, d], bufs["lse"] [P, Hq, n].  Returns the milliseconds of the whole
        program when ``timed``."""
        if not self.planned:
            raise RuntimeError("call plan() first")
        P = self.P
        main = torch.cuda.current_stream()
        streams = [torch.cuda.Stream(device=self.device) for _ in range(P)]
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(main)
        done = [start] * P      # the event each rank's stream must pass before the next stage
        by_stage = [[[] for _ in range(self.num_stages)] for _ in range(P)]
        for e in range(P):
            for o in self.ops[e]:
                by_stage[e][int(o[3])].append([int(x) for x in o])
        for t in range(self.num_stages):
            stage_done = []
            for e in range(P):
                s = streams[e]
                for ev in set(done):
                    s.wait_event(ev)
                with torch.cuda.stream(s):
                    for op, tensor, peer, _, shard, chunk, in_slot, out_slot in by_stage[e][t]:
                        if op == L.OP_RECV:
                            if tensor == L.T_Q:
                                bufs["q_recv"][e][out_slot].copy_(q[peer])
                            elif tensor == L.T_KV:
                                bufs["k_recv"][e][out_slot].copy_(k[peer])
                                bufs["v_recv"][e][out_slot].copy_(v[peer])
                            else:
                                src = self._send_slot(peer, e, t, shard, chunk)
                                bufs["o_part"][e][out_slot].copy_(bufs["o_res"][peer][src])
                                bufs["lse_part"][e][out_slot].copy_(bufs["lse_res"][peer][src])
                        elif op == L.OP_COMPUTE:
                            qq = q[e] if shard == e else bufs["q_recv"][e][in_slot]
                            # the own chunk, or the receive slot holding chunk `chunk` alone
                            kk, vv = k[chunk], v[chunk]
                            if chunk != e:
                                kk, vv = bufs["k_recv"][e][in_slot], bufs["v_recv"][e][in_slot]
                            if shard == e:
                                ob, lb = bufs["o_part"][e], bufs["lse_part"][e]
                            else:
                                ob, lb = bufs["o_res"][e], bufs["lse_res"][e]
                            L.partial_attn_fwd_runs(self.descs[shard], qq, kk, vv, self.doc_start, self.tiles_dev[shard],
                                               self._runs(shard, chunk, out_slot), ob, lb, stream=s, kv_chunk=chunk)
                        elif op == L.OP_MERGE:
                            parts = out_slot
                            L.lse_merge([bufs["o_part"][e][i] for i in range(parts)],
                                        [bufs["lse_part"][e][i] for i in range(parts)], self.n, self.hq, self.d,
                                        bufs["o"][e], bufs["lse"][e], stream=s)
                ev = torch.cuda.Event()
                ev.record(s)
                stage_done.append(ev)
            done = stage_done
        for ev in done:
            main.wait_event(ev)
        end.record(main)
        if not timed:
            return None
        end.synchronize()
        return start.elapsed_time(end)

    def _send_slot(self, sender: int, receiver: int, stage: int, shard: int, chunk: int, tensor: int = L.T_O,
                   ops=None) -> int:
        for o in (self.ops if ops is None else ops)[sender]:
            if (int(o[0]) == L.OP_SEND and int(o[1]) == tensor and int(o[2]) == receiver and int(o[3]) == stage
                    and int(o[4]) == shard and int(o[5]) == chunk):
                return int(o[6])
        raise RuntimeError("no matching send for a receive of tensor %d" % tensor)

    # ------------------------------------------------------------------ backward
    def alloc_backward(self) -> Dict[str, list]:
        P, n, dev = self.P, self.n, self.device
        bf, f32 = torch.bfloat16, torch.float32
        hq, hkv, d = self.hq, self.hkv, self.d
        return {
            "delta": torch.empty(P, hq, n, dtype=f32, device=dev),
            "q_recv": [torch.empty(2, n, hq, d, dtype=bf, device=dev) for _ in range(P)],
            "do_recv": [torch.empty(2, n, hq, d, dtype=bf, device=dev) for _ in range(P)],
            "lse_recv": [torch.empty(2, hq, n, dtype=f32, device=dev) for _ in range(P)],
            "delta_recv": [torch.empty(2, hq, n, dtype=f32, device=dev) for _ in range(P)],
            "k_recv": [torch.empty(2, n, hkv, d, dtype=bf, device=dev) for _ in range(P)],
            "v_recv": [torch.empty(2, n, hkv, d, dtype=bf, device=dev) for _ in range(P)],
            "dq_res": [torch.empty(2, n, hq, d, dtype=f32, device=dev) for _ in range(P)],
            "dk_res": [torch.empty(2, n, hkv, d, dtype=f32, device=dev) for _ in range(P)],
            "dv_res": [torch.empty(2, n, hkv, d, dtype=f32, device=dev) for _ in range(P)],
            "dq_part": [torch.empty(max(len(x), 1), n, hq, d, dtype=f32, device=dev) for x in self.dq_parts],
            "dk_part": [torch.empty(max(len(x), 1), n, hkv, d, dtype=f32, device=dev) for x in self.dkv_parts],
            "dv_part": [torch.empty(max(len(x), 1), n, hkv, d, dtype=f32, device=dev) for x in self.dkv_parts],
            "dq": torch.empty(P, n, hq, d, dtype=bf, device=dev),
            "dk": torch.empty(P, n, hkv, d, dtype=bf, device=dev),
            "dv": torch.empty(P, n, hkv, d, dtype=bf, device=dev),
        }

    def run_backward(self, q, k, v, d_o, o, lse, bufs: Dict[str, list], timed: bool = False) -> Optional[float]:
        """q, d_o, o [P, n, Hq, d] and lse [P, Hq, n] (every rank's shard: inputs, output gradient, the
        forward's output and LSE), k / v [P, n, Hkv, d] -> bufs["dq"] [P, n, Hq, d], bufs["dk"] /
        bufs["dv"] [P, n, Hkv, d] (bf16; chunks without any block stay as they are).  Returns the
        milliseconds of the whole program when ``timed``."""
        if not (self.planned and self.backward_planned):
            raise RuntimeError("call plan(backward=True) first")
        P, ops = self.P, self.ops_bwd
        main = torch.cuda.current_stream()
        streams = [torch.cuda.Stream(device=self.device) for _ in range(P)]
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(main)
        by_stage = [[[] for _ in range(self.num_stages_bwd)] for _ in range(P)]
        for e in range(P):
            for op in ops[e]:
                by_stage[e][int(op[3])].append([int(x) for x in op])
        # before stage 0: each rank's own row term delta = rowsum(dO o O)
        done = []
        for e in range(P):
            streams[e].wait_event(start)
            with torch.cuda.stream(streams[e]):
                L.attn_bwd_preprocess(o[e], d_o[e], self.n, self.hq, self.d, bufs["delta"][e], stream=streams[e])
            ev = torch.cuda.Event()
            ev.record(streams[e])
            done.append(ev)
        for t in range(self.num_stages_bwd):
            stage_done = []
            for e in range(P):
                s = streams[e]
                for ev in set(done):
                    s.wait_event(ev)
                with torch.cuda.stream(s):
                    for op, tensor, peer, _, shard, chunk, in_slot, out_slot in by_stage[e][t]:
                        if op == L.OP_RECV:
                            self._receive_backward(bufs, e, t, tensor, peer, shard, chunk, out_slot, q, d_o, lse,
                                                   k, v)
                        elif op == L.OP_COMPUTE:
                            self._compute_backward(bufs, e, shard, chunk, in_slot, out_slot, q, d_o, lse, k, v, s)
                        elif op == L.OP_MERGE and tensor == L.T_DQ:
                            L.sum_parts([bufs["dq_part"][e][i] for i in range(out_slot)], bufs["dq"][e], stream=s)
                        elif op == L.OP_MERGE:
                            L.sum_parts([bufs["dk_part"][e][i] for i in range(out_slot)], bufs["dk"][e], stream=s)
                            L.sum_parts([bufs["dv_part"][e][i] for i in range(out_slot)], bufs["dv"][e], stream=s)
                ev = torch.cuda.Event()
                ev.record(s)
                stage_done.append(ev)
            done = stage_done
        for ev in done:
            main.wait_event(ev)
        end.record(main)
        if not timed:
            return None
        end.synchronize()
        return start.elapsed_time(end)

    def _receive_backward(self, bufs, e, t, tensor, peer, shard, chunk, out_slot, q, d_o, lse, k, v) -> None:
        """A receive of the backward program: a device copy out of the sending rank's buffer."""
        if tensor == L.T_Q:
            bufs["q_recv"][e][out_slot].copy_(q[peer])
        elif tensor == L.T_DO:
            bufs["do_recv"][e][out_slot].copy_(d_o[peer])
            bufs["lse_recv"][e][out_slot].copy_(lse[peer])
            bufs["delta_recv"][e][out_slot].copy_(bufs["delta"][peer])
        elif tensor == L.T_KV:
            bufs["k_recv"][e][out_slot].copy_(k[peer])
            bufs["v_recv"][e][out_slot].copy_(v[peer])
        elif tensor == L.T_DQ:
            src = self._send_slot(peer, e, t, shard, chunk, L.T_DQ, self.ops_bwd)
            bufs["dq_part"][e][out_slot].copy_(bufs["dq_res"][peer][src])
        else:
            src = self._send_slot(peer, e, t, shard, chunk, L.T_DKV, self.ops_bwd)
            bufs["dk_part"][e][out_slot].copy_(bufs["dk_res"][peer][src])
            bufs["dv_part"][e][out_slot].copy_(bufs["dv_res"][peer][src])

    def _compute_backward(self, bufs, e, r, c, in_slot, out_slot, q, d_o, lse, k, v, stream) -> None:
        """Block (r, c) on rank e: its dQ part and dK/dV part, each into the rank's own part buffer
        or into the result slot it is sent from."""
        if r == e:
            qq, dd, ll, de = q[e], d_o[e], lse[e], bufs["delta"][e]
            dq_t = bufs["dq_part"][e][self.dq_parts[e].index(c)]
        else:
            qq, dd = bufs["q_recv"][e][in_slot], bufs["do_recv"][e][in_slot]
            ll, de = bufs["lse_recv"][e][in_slot], bufs["delta_recv"][e][in_slot]
            dq_t = bufs["dq_res"][e][out_slot]
        if c == e:
            kk, vv = k[e], v[e]
            dk_t = bufs["dk_part"][e][self.dkv_parts[e].index(r)]
            dv_t = bufs["dv_part"][e][self.dkv_parts[e].index(r)]
        else:
            kk, vv = bufs["k_recv"][e][in_slot], bufs["v_recv"][e][in_slot]
            dk_t, dv_t = bufs["dk_res"][e][out_slot], bufs["dv_res"][e][out_slot]
        for t_ in (dq_t, dk_t, dv_t):
            t_.zero_()
        L.partial_attn_bwd_runs(self.descs[r], qq, kk, vv, dd, ll, de, self.doc_start, self.tiles_k_dev[r],
                           self._runs_k(r, c), self.tiles_dev[r], self._runs(r, c, c), dq_t, dk_t, dv_t,
                           stream=stream, kv_chunk=c)
