"""Which global token positions each sequence-parallel shard holds (oracle side).

Inter-group sequence parallelism cuts the packed sequence of N tokens along
its length into P blocks of n = N / P tokens, one per rank (inter-group SP
section; the HSAP hierarchy section cuts the same way before splitting heads).

* contiguous: shard r holds positions r*n .. r*n + n - 1.
* zigzag: the sequence is cut into 2P equal pieces of m = N / (2P) tokens and
  shard r holds piece r followed by piece 2P-1-r.  The paper does not spell
  this layout out; it delegates ring load balancing to LightSeq.  Under it,
  one causal document spanning the whole sequence gives every shard the same
  number of query-key pairs.

A shard's K/V chunk has the same layout as its queries.  In ring order, shard
r holds chunk (r - s) mod P at ring step s (each rank passes K/V to its
neighbour after every step).
"""
from __future__ import annotations

import numpy as np


def shard_positions(total_tokens: int, sp_degree: int, layout: str, shard: int) -> np.ndarray:
    """Global positions (int64) of shard ``shard``'s local rows, in local order."""
    N, P = int(total_tokens), int(sp_degree)
    if not (0 <= shard < P):
        raise ValueError("shard out of range")
    if layout == "contiguous":
        if N % P:
            raise ValueError("N must be divisible by P")
        n = N // P
        return np.arange(shard * n, (shard + 1) * n, dtype=np.int64)
    if layout == "zigzag":
        if N % (2 * P):
            raise ValueError("N must be divisible by 2P")
        m = N // (2 * P)
        first = np.arange(shard * m, (shard + 1) * m, dtype=np.int64)
        second_piece = 2 * P - 1 - shard
        second = np.arange(second_piece * m, (second_piece + 1) * m, dtype=np.int64)
        return np.concatenate([first, second])
    raise ValueError("unknown layout %r" % (layout,))


def ring_chunk(shard: int, step: int, sp_degree: int) -> int:
    """Chunk held by ``shard`` at ring step ``step``: (shard - step) mod P."""
    return (shard - step) % sp_degree
