"""Per-rank instruction lists of the forward and backward passes (the jitted code of the SAP section).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The instruction set is the paper's (instruction table of the SAP section):
send and receive of q, kv or o to or from a peer rank, computing on the
tensors in the computing buffer, and local copies between buffers; the last
compile step turns the block layout into one such list per rank, arranged in
stages so that each stage's transfers (data for the next stage, results of
the previous one) run beside its computation, with every send matched by the
receive at the same position of the peer's list.  The paper gives no
concrete arrangement; the reading used here (each step written in the order
below):

* Rank e computes the non-empty blocks (r, c) assigned to it, one per stage:
  its diagonal block (e, e) first (local data only), then the others ordered
  by ring step (r - c) mod P, then r, then c.  A rank without a diagonal block
  starts at stage 1 (its first input must arrive first).  S = one past the
  last compute stage of any rank; stage S only returns results and merges.
* Inputs arrive one stage ahead, straight from their owner (every rank owns
  its Q shard and its K/V chunk): for block (e, c) at stage t, rank c sends kv
  (chunk c) to e at stage t-1; for a transferred block (r, e), rank r sends q
  (shard r) to e at stage t-1.  The receiver keeps them in slot t % 2 of its
  receive buffers (two slots per kind: a stage's receives never touch what
  its computation reads).
* A transferred block's partial (o and its log-sum-exp) is written to slot
  t % 2 of the computing rank's result buffer at stage t and sent to r at
  stage t+1, where r keeps it as the part of chunk c.
* After its last receive, rank r merges its parts (the separate copy and
  rescale of partial outputs, done here as one merge of every part).
* Parts of shard r are the chunks with a non-empty block (r, c), in
  increasing chunk order; part(r, c) is c's index among them.
* Within a stage a rank lists its sends and receives first, ordered by
  (peer, kind with send before receive, tensor, shard, chunk), then its
  computation, then the merge.

The backward program (``backward_program``) moves the gradient messages of
the same instruction table (dq, dkv, do).  Reading:

* Every block is differentiated on the rank that computed its forward, at the
  same stage as there (the forward's block order and first stages).
* A ring block (r, c), c != r, on rank r: chunk c's K/V come from rank c one
  stage ahead into receive slot t % 2 (as in the forward).  Its dQ part stays
  on r; its dK/dV part is written to result slot t % 2 and sent to rank c at
  stage t+1 as tensor dkv.
* A transferred block (r, c) on rank c: shard r's Q and its dO (with the
  shard's final LSE and delta) come from rank r at stage t-1 into receive slot
  t % 2, as two messages (q, then do).  Its dK/dV part stays on c; its dQ
  part goes to result slot t % 2 and is sent to rank r at stage t+1 as tensor
  dq.
* A diagonal block keeps both parts.
* COMPUTE carries in_slot = receive slot and out_slot = result slot (both -1
  for a diagonal block).  Parts that stay and parts received are indexed by
  kind: dQ parts of shard r by chunk (index of c among the chunks with a
  block of shard r), dK/dV parts of chunk c by shard (index of r among the
  shards with a block in chunk c); a receive names that index in out_slot.
* In the last stage each rank sums its dQ parts in index order (MERGE of
  tensor dq, shard e, out_slot = count) and then its dK/dV parts (MERGE of
  tensor dkv, chunk e, out_slot = count) -- the accumulation the paper does
  with local copies into its gradient buffers.
* Order within a stage: as in the forward.

Op tuples: (op, tensor, peer, stage, shard, chunk, in_slot, out_slot), the
fields of the library's op record.  Pins: ``tests/test_schedule.py`` checks
matched sends and receives, that every block is computed once on its rank
with inputs that arrived earlier, slot lifetimes, and runs the lists on fp64
data through ``attention.attention_fwd`` / ``attention.lse_merge`` to the
per-shard result of ``attention.shard_forward``.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

OP_SEND, OP_RECV, OP_COMPUTE, OP_MERGE = 0, 1, 2, 3
T_NONE, T_Q, T_KV, T_O, T_DQ, T_DKV, T_DO = -1, 0, 1, 2, 3, 4, 5

Op = Tuple[int, int, int, int, int, int, int, int]


def forward_program(block_tiles, exec_rank) -> Tuple[List[List[Op]], int]:
    """(ops per rank, number of stages) for block sizes [P, P] and their ranks [P, P]."""
    tiles = np.asarray(block_tiles, dtype=np.int64)
    ex = np.asarray(exec_rank, dtype=np.int64)
    P = tiles.shape[0]
    # blocks per rank, in stage order
    blocks = [[] for _ in range(P)]
    for r in range(P):
        for c in range(P):
            if tiles[r, c] > 0:
                blocks[int(ex[r, c])].append((r, c))
    for e in range(P):
        blocks[e].sort(key=lambda b: (0 if b[0] == b[1] else 1, (b[0] - b[1]) % P, b[0], b[1]))
    first = [0 if blocks[e] and blocks[e][0][0] == blocks[e][0][1] else 1 for e in range(P)]
    S = max(first[e] + len(blocks[e]) for e in range(P))
    parts = [[c for c in range(P) if tiles[r, c] > 0] for r in range(P)]

    def part(r, c):
        return parts[r].index(c)

    comm = [[[] for _ in range(S + 1)] for _ in range(P)]
    compute = [[[] for _ in range(S + 1)] for _ in range(P)]
    for e in range(P):
        for i, (r, c) in enumerate(blocks[e]):
            t = first[e] + i
            if r == e and c != e:          # K/V of chunk c from its owner, one stage ahead
                comm[c][t - 1].append((OP_SEND, T_KV, e, t - 1, -1, c, -1, -1))
                comm[e][t - 1].append((OP_RECV, T_KV, c, t - 1, -1, c, -1, t % 2))
            elif c == e and r != e:        # Q of shard r from its owner, one stage ahead
                comm[r][t - 1].append((OP_SEND, T_Q, e, t - 1, r, -1, -1, -1))
                comm[e][t - 1].append((OP_RECV, T_Q, r, t - 1, r, -1, -1, t % 2))
                # the partial goes back one stage later
                comm[e][t + 1].append((OP_SEND, T_O, r, t + 1, r, c, t % 2, -1))
                comm[r][t + 1].append((OP_RECV, T_O, e, t + 1, r, c, -1, part(r, c)))
            in_slot = -1 if r == c else t % 2
            out_slot = part(r, c) if r == e else t % 2
            compute[e][t].append((OP_COMPUTE, T_NONE, -1, t, r, c, in_slot, out_slot))
    program = []
    for e in range(P):
        ops = []
        for t in range(S + 1):
            ops += sorted(comm[e][t], key=lambda o: (o[2], o[0], o[1], o[4], o[5]))
            ops += compute[e][t]
            if t == S and parts[e]:
                ops.append((OP_MERGE, T_NONE, -1, S, e, -1, -1, len(parts[e])))
        program.append(ops)
    return program, S + 1


def backward_program(block_tiles, exec_rank) -> Tuple[List[List[Op]], int]:
    """(ops per rank, number of stages) of the backward pass for block sizes [P, P] and ranks [P, P]."""
    tiles = np.asarray(block_tiles, dtype=np.int64)
    ex = np.asarray(exec_rank, dtype=np.int64)
    P = tiles.shape[0]
    # the forward's stage of every block
    on_rank = [[] for _ in range(P)]
    for r in range(P):
        for c in range(P):
            if tiles[r, c] > 0:
                on_rank[int(ex[r, c])].append((r, c))
    for e in range(P):
        on_rank[e].sort(key=lambda b: (b[0] != b[1], (b[0] - b[1]) % P, b[0], b[1]))
    start = [0 if on_rank[e] and on_rank[e][0][0] == on_rank[e][0][1] else 1 for e in range(P)]
    last = max(start[e] + len(on_rank[e]) for e in range(P))
    dq_parts = [[c for c in range(P) if tiles[r, c] > 0] for r in range(P)]      # of shard r, by chunk
    dkv_parts = [[r for r in range(P) if tiles[r, c] > 0] for c in range(P)]     # of chunk c, by shard

    transfers = [[[] for _ in range(last + 1)] for _ in range(P)]
    work = [[[] for _ in range(last + 1)] for _ in range(P)]
    for e in range(P):
        for k, (r, c) in enumerate(on_rank[e]):
            t = start[e] + k
            slot = t % 2
            if r == c:
                work[e][t].append((OP_COMPUTE, T_NONE, -1, t, r, c, -1, -1))
                continue
            if r == e:       # ring block: K/V in; dK/dV out to the chunk's owner
                transfers[c][t - 1].append((OP_SEND, T_KV, e, t - 1, -1, c, -1, -1))
                transfers[e][t - 1].append((OP_RECV, T_KV, c, t - 1, -1, c, -1, slot))
                transfers[e][t + 1].append((OP_SEND, T_DKV, c, t + 1, r, c, slot, -1))
                transfers[c][t + 1].append((OP_RECV, T_DKV, e, t + 1, r, c, -1, dkv_parts[c].index(r)))
            else:            # transferred block: Q and dO in; dQ out to the shard's owner
                for tensor in (T_Q, T_DO):
                    transfers[r][t - 1].append((OP_SEND, tensor, e, t - 1, r, -1, -1, -1))
                    transfers[e][t - 1].append((OP_RECV, tensor, r, t - 1, r, -1, -1, slot))
                transfers[e][t + 1].append((OP_SEND, T_DQ, r, t + 1, r, c, slot, -1))
                transfers[r][t + 1].append((OP_RECV, T_DQ, e, t + 1, r, c, -1, dq_parts[r].index(c)))
            work[e][t].append((OP_COMPUTE, T_NONE, -1, t, r, c, slot, slot))
    program = []
    for e in range(P):
        ops = []
        for t in range(last + 1):
            ops += sorted(transfers[e][t], key=lambda o: (o[2], o[0], o[1], o[4], o[5]))
            ops += work[e][t]
            if t == last:
                if dq_parts[e]:
                    ops.append((OP_MERGE, T_DQ, -1, last, e, -1, -1, len(dq_parts[e])))
                if dkv_parts[e]:
                    ops.append((OP_MERGE, T_DKV, -1, last, -1, e, -1, len(dkv_parts[e])))
        program.append(ops)
    return program, last + 1
