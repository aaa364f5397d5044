"""Tile classification of one shard's attention against every K/V chunk (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The compile step of SAP first cuts the packed causal mask into per-rank blocks
and sorts each block by its attention pattern (compile step 1 of the SAP
section; the pattern figure itself is missing from the text).  Here the same
partition is taken one level finer: shard r's n query rows are cut into
q-tiles of BM rows, chunk c's n key rows into k-tiles of BN rows, and every
(q-tile, k-tile) pair is classified by how many of its BM*BN (query, key)
pairs the packing mask allows:

  * EMPTY  -- none (never listed, never computed);
  * FULL   -- all BM*BN (kind 0: no masking needed);
  * MASKED -- some but not all (kind 1: the mask is applied per element).

Canonical order (needed for a bit-exact list): ring step ascending (step s
holds chunk (r - s) mod P), then q-tile ascending, then k-tile ascending.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .attention import allowed_mask_dense, doc_starts
from .layout import ring_chunk, shard_positions

KIND_FULL = 0
KIND_MASKED = 1


def tile_pair_counts_bruteforce(cu_seqlens, total_tokens, sp_degree, layout, shard, chunk,
                                block_m, block_n) -> np.ndarray:
    """Allowed-pair count of every (q-tile, k-tile), by classifying each pair.

    Builds the dense mask pair by pair from document ids; tiny inputs only.
    Returns int64 [n/BM, n/BN].
    """
    q_pos = shard_positions(total_tokens, sp_degree, layout, shard)
    k_pos = shard_positions(total_tokens, sp_degree, layout, chunk)
    mask = allowed_mask_dense(cu_seqlens, q_pos, k_pos)
    n = len(q_pos)
    return mask.reshape(n // block_m, block_m, n // block_n, block_n).sum(axis=(1, 3)).astype(np.int64)


def tile_pair_counts(cu_seqlens, total_tokens, sp_degree, layout, shard, chunk,
                     block_m, block_n) -> np.ndarray:
    """Allowed-pair count of every (q-tile, k-tile), counted row by row.

    For query row i with start s_i and position p_i, the keys of a k-tile it
    may attend to are those with s_i <= position <= p_i; their number is read
    off the tile's sorted key positions with two binary searches.  Summing the
    row counts over a q-tile's rows gives the tile count.  Returns int64
    [n/BM, n/BN].
    """
    q_pos = shard_positions(total_tokens, sp_degree, layout, shard)
    k_pos = shard_positions(total_tokens, sp_degree, layout, chunk)
    n = len(q_pos)
    if n % block_m or n % block_n:
        raise ValueError("tile sizes must divide the shard length")
    starts = doc_starts(cu_seqlens)
    s_i = starts[q_pos]
    nq_t, nk_t = n // block_m, n // block_n
    out = np.zeros((nq_t, nk_t), dtype=np.int64)
    for u in range(nk_t):
        kp = np.sort(k_pos[u * block_n:(u + 1) * block_n])
        row_counts = (np.searchsorted(kp, q_pos, side="right")
                      - np.searchsorted(kp, s_i, side="left"))
        row_counts = np.maximum(row_counts, 0)
        out[:, u] = row_counts.reshape(nq_t, block_m).sum(axis=1)
    return out


def plan_shard(cu_seqlens, total_tokens, sp_degree, layout, shard, block_m, block_n,
               counter=tile_pair_counts) -> Dict:
    """Non-empty tiles of shard ``shard`` in canonical order.

    Returns a dict with
      ``tiles``        int32 [T, 4] rows (chunk, q_tile, k_tile, kind),
      ``pairs``        int64 [T] allowed pairs of each listed tile,
      ``step_offsets`` int64 [P+1] CSR offsets of each ring step's tiles,
      ``useful_pairs`` int64 [P] allowed pairs per ring step.
    """
    full = block_m * block_n
    tiles, pairs, offsets, useful = [], [], [0], []
    for step in range(sp_degree):
        c = ring_chunk(shard, step, sp_degree)
        counts = counter(cu_seqlens, total_tokens, sp_degree, layout, shard, c, block_m, block_n)
        step_pairs = 0
        for t in range(counts.shape[0]):
            for u in range(counts.shape[1]):
                cnt = int(counts[t, u])
                if cnt == 0:
                    continue
                tiles.append((c, t, u, KIND_FULL if cnt == full else KIND_MASKED))
                pairs.append(cnt)
                step_pairs += cnt
        offsets.append(len(tiles))
        useful.append(step_pairs)
    return {
        "tiles": np.asarray(tiles, dtype=np.int32).reshape(-1, 4),
        "pairs": np.asarray(pairs, dtype=np.int64),
        "step_offsets": np.asarray(offsets, dtype=np.int64),
        "useful_pairs": np.asarray(useful, dtype=np.int64),
    }


def useful_pairs_all_shards(cu_seqlens, total_tokens, sp_degree, layout) -> np.ndarray:
    """Allowed (query, key) pairs of every shard over all chunks (int64 [P]).

    The chunks together hold every position, so a query at position i with
    start s contributes exactly i - s + 1 keys.
    """
    starts = doc_starts(cu_seqlens)
    out = np.zeros(sp_degree, dtype=np.int64)
    for r in range(sp_degree):
        q_pos = shard_positions(total_tokens, sp_degree, layout, r)
        out[r] = int(np.sum(q_pos - starts[q_pos] + 1))
    return out
