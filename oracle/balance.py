"""Per-(shard, chunk) load of a packed sequence and the Q-transfer rebalance.

TEST INFRASTRUCTURE ONLY (see the package docstring): nothing on the product
path imports this module.

* ``load_matrix`` -- the size of every rank block of the compile step's block
  partition (compile step 1 of the SAP section): for shard r (query rows) and
  chunk c (key rows), the number of non-empty BM x BN tiles and of allowed
  (query, key) pairs, taken from the per-shard plan of ``plan.plan_shard``.
* ``q_transfer_balance`` -- the workload balancing of compile step 2, which the
  paper bases on LightSeq's scheduling and which it states as balancing the
  number of attention blocks each rank computes, together with the balancing
  of InterSP groups by additionally transferring Q blocks (memory and
  communication section).  The paper gives no algorithm; the reading used
  here: a block (r, c) with r != c runs either on rank r once chunk c's K/V
  reach it (the ring), or on rank c, the owner of chunk c, once Q_r reaches it
  (its partial O and LSE then travel back to r for the merge).  Diagonal
  blocks stay on their rank.  Starting from the ring assignment, the most
  loaded rank (lowest index among equals) hands one of its blocks to that
  block's other eligible rank, as long as the receiver stays below the giver's
  current load; among such moves the one leaving the smaller of the two new
  loads' maximum is taken (equal: lower r, then lower c).  It stops when the
  most loaded rank has no such move.  Every move lowers the sum of squared
  loads, so it ends.

Pins (``tests/test_oracle_pins.py``): pair counts against the dense mask and
the closed-form per-shard total; the assignment against brute force over every
assignment on small matrices (and equality where one block is movable), its
invariants, and a worked example.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from .layout import ring_chunk
from .plan import plan_shard


def load_matrix(cu_seqlens, total_tokens: int, sp_degree: int, layout: str, block_m: int,
                block_n: int) -> Tuple[np.ndarray, np.ndarray]:
    """(tiles, pairs), both int64 [P, P] indexed [shard r, chunk c]."""
    P = sp_degree
    tiles = np.zeros((P, P), dtype=np.int64)
    pairs = np.zeros((P, P), dtype=np.int64)
    for r in range(P):
        plan = plan_shard(cu_seqlens, total_tokens, P, layout, r, block_m, block_n)
        for step in range(P):
            c = ring_chunk(r, step, P)
            tiles[r, c] = plan["step_offsets"][step + 1] - plan["step_offsets"][step]
            pairs[r, c] = plan["useful_pairs"][step]
    return tiles, pairs


def q_transfer_balance(cost) -> Tuple[np.ndarray, np.ndarray]:
    """(exec_rank int32 [P, P], load int64 [P]) for block costs ``cost`` [P, P].

    exec_rank[r, c] is the rank that computes shard r's queries against chunk
    c: r (ring delivery of K/V) or c (Q transfer).  Empty blocks keep r.
    """
    cost = np.asarray(cost, dtype=np.int64)
    P = cost.shape[0]
    exec_rank = np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
    load = [int(cost[r].sum()) for r in range(P)]
    while True:
        giver = max(range(P), key=lambda e: (load[e], -e))      # most loaded, lowest index among equals
        best = None
        for r in range(P):
            for c in range(P):
                w = int(cost[r, c])
                if r == c or w == 0 or giver not in (r, c) or exec_rank[r, c] != giver:
                    continue
                taker = c if giver == r else r
                if load[taker] + w >= load[giver]:
                    continue
                key = (max(load[giver] - w, load[taker] + w), r, c)
                if best is None or key < best[0]:
                    best = (key, r, c, taker, w)
        if best is None:
            break
        _, r, c, taker, w = best
        exec_rank[r, c] = taker
        load[giver] -= w
        load[taker] += w
    return exec_rank, np.asarray(load, dtype=np.int64)
