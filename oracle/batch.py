"""Batches of packed sequences: B sequences of N tokens, concatenated, each sharded P ways.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A batch is B independent packed sequences: attention never crosses a sequence
(every sequence start is a document boundary), so every result is the
single-sequence result of each sequence, placed at its rows.  Shard x's local
rows over the batch are b*n + l (row l of sequence b, n = N/P), its q-tiles
b*(n/BM) + t and a chunk's k-tiles b*(n/BN) + u.  These functions compute
exactly that with the single-sequence oracle, one sequence at a time.

Pins (``tests/test_oracle_pins.py``): a batch of one sequence equals the
single-sequence call; a batch of copies gives copies; the tile list of a batch
equals the brute-force classification of the concatenated sequence's pairs
restricted to the shard's rows.
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from .attention import shard_backward, shard_forward
from .plan import plan_shard


def split_batch(cu_seqlens, total_tokens: int, batch: int) -> List[np.ndarray]:
    """Per-sequence cumulative lengths (each starting at 0) of a batch's concatenated cu_seqlens."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = []
    for b in range(batch):
        lo, hi = b * total_tokens, (b + 1) * total_tokens
        if lo not in cu or hi not in cu:
            raise ValueError("every sequence start must be a document boundary")
        seg = cu[(cu >= lo) & (cu <= hi)] - lo
        out.append(np.unique(seg))
    return out


def batch_plan_shard(cu_seqlens, total_tokens: int, batch: int, sp_degree: int, layout: str, shard: int,
                     block_m: int, block_n: int) -> Dict:
    """Non-empty tiles of shard ``shard`` over the batch, canonical order (ring step, q-tile, k-tile)."""
    n = total_tokens // sp_degree
    plans = [plan_shard(cu_b, total_tokens, sp_degree, layout, shard, block_m, block_n)
             for cu_b in split_batch(cu_seqlens, total_tokens, batch)]
    tiles, offsets, useful = [], [0], []
    for step in range(sp_degree):
        count, pairs = 0, 0
        for b, p in enumerate(plans):
            seg = p["tiles"][p["step_offsets"][step]:p["step_offsets"][step + 1]].copy()
            seg[:, 1] += b * (n // block_m)
            seg[:, 2] += b * (n // block_n)
            tiles.append(seg)
            count += len(seg)
            pairs += int(p["useful_pairs"][step])
        offsets.append(offsets[-1] + count)
        useful.append(pairs)
    return {"tiles": np.concatenate(tiles).astype(np.int32).reshape(-1, 4),
            "step_offsets": np.asarray(offsets, dtype=np.int64),
            "useful_pairs": np.asarray(useful, dtype=np.int64)}


def batch_shard_forward(q, k, v, cu_seqlens, total_tokens: int, batch: int, sp_degree: int, layout: str,
                        shard: int) -> Dict:
    """Merged O [B*n, Hq, d] and LSE [Hq, B*n] of shard ``shard`` over the batch (q, k, v in
    concatenated global order, [B*N, ...])."""
    N = total_tokens
    os_, lses = [], []
    for b, cu_b in enumerate(split_batch(cu_seqlens, N, batch)):
        sl = slice(b * N, (b + 1) * N)
        res = shard_forward(q[sl], k[sl], v[sl], cu_b, N, sp_degree, layout, shard)
        os_.append(res["o"])
        lses.append(res["lse"])
    return {"o": np.concatenate(os_, axis=0), "lse": np.concatenate(lses, axis=1)}


def batch_shard_backward(q, k, v, d_o, cu_seqlens, total_tokens: int, batch: int, sp_degree: int, layout: str,
                         shard: int) -> Dict:
    """dQ [B*n, Hq, d] of shard ``shard`` and its dK / dV contributions [P, B*n, Hkv, d] (chunk c's
    rows b*n + l) over the batch."""
    N, P = total_tokens, sp_degree
    dq, dk, dv = [], [], []
    for b, cu_b in enumerate(split_batch(cu_seqlens, N, batch)):
        sl = slice(b * N, (b + 1) * N)
        res = shard_backward(q[sl], k[sl], v[sl], d_o[sl], cu_b, N, P, layout, shard)
        dq.append(res["dq"])
        dk.append(res["dk"])
        dv.append(res["dv"])
    return {"dq": np.concatenate(dq, axis=0), "dk": np.concatenate(dk, axis=1), "dv": np.concatenate(dv, axis=1)}
