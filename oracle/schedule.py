"""Per-rank instruction lists of the forward pass (the jitted code of the SAP section).

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
T_NONE, T_Q, T_KV, T_O = -1, 0, 1, 2

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
