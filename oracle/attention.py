"""fp64 reference for document-masked causal attention, its partials, merge and gradients.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Conventions (each is a reading of the paper, which is silent on them):
  * positions are global token indices 0 .. N-1 of the packed sequence;
  * start(t) is the first position of t's document; a query at position i may
    attend to a key at position j iff start(i) <= j <= i (same document,
    causal, diagonal included);
  * query head h reads key/value head h // (Hq / Hkv) (grouped-query
    attention with contiguous groups; the paper itself only has Hq = Hkv);
  * softmax scale 1/sqrt(d) unless given; LSE is the natural-log log-sum-exp
    of the scaled scores over the allowed keys, laid out [Hq, rows];
  * a row with no allowed key has O = 0 and LSE = -inf.

All arithmetic is float64.  Inputs may be any real arrays (the tests pass the
bf16-rounded values); they are promoted to float64 here.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np

from .layout import ring_chunk, shard_positions


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def doc_starts(cu_seqlens) -> np.ndarray:
    """start(t) for every position t of the packed sequence (int64 [N]).

    ``cu_seqlens`` holds the cumulative document lengths (first entry 0, last
    entry N); document k covers positions cu[k] .. cu[k+1]-1.
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    lengths = np.diff(cu)
    if cu[0] != 0 or np.any(lengths < 0):
        raise ValueError("cu_seqlens must start at 0 and be non-decreasing")
    return np.repeat(cu[:-1], lengths)


def allowed_mask_dense(cu_seqlens, q_pos: Sequence[int], k_pos: Sequence[int]) -> np.ndarray:
    """Boolean [len(q_pos), len(k_pos)] mask built pair by pair from document ids.

    This is the mask written the other way round from ``attention_fwd``: two
    positions may interact iff they lie in the same document and the key does
    not come after the query.  Meant for tiny inputs only.
    """
    cu = [int(c) for c in cu_seqlens]

    def doc_of(t: int) -> int:
        for d in range(len(cu) - 1):
            if cu[d] <= t < cu[d + 1]:
                return d
        raise ValueError("position outside the packed sequence")

    qd = [doc_of(int(i)) for i in q_pos]
    kd = [doc_of(int(j)) for j in k_pos]
    out = np.zeros((len(q_pos), len(k_pos)), dtype=bool)
    for a, i in enumerate(q_pos):
        for b, j in enumerate(k_pos):
            out[a, b] = (qd[a] == kd[b]) and (int(j) <= int(i))
    return out


def _row_blocks(q_pos: np.ndarray, q_start: np.ndarray, row_block: int):
    """Yield index arrays of query rows that share one document, in position order."""
    order = np.argsort(q_pos, kind="stable")
    i, nq = 0, len(order)
    while i < nq:
        s = q_start[order[i]]
        j = i + 1
        while j < nq and j - i < row_block and q_start[order[j]] == s:
            j += 1
        yield int(s), order[i:j]
        i = j


def attention_fwd(q, k, v, q_pos, k_pos, cu_seqlens, scale: Optional[float] = None,
                  row_block: int = 256):
    """Masked attention of query rows against a set of key/value rows.

    q: [nq, Hq, d]; k, v: [nk, Hkv, d]; q_pos: [nq] and k_pos: [nk] global
    positions of those rows.  Returns (O [nq, Hq, d], LSE [Hq, nq]).

    Only the keys inside the query's own document and not after it contribute
    (the packing mask); O is the softmax-weighted sum of their values with the
    scores q.k * scale (the attention equation), LSE the log of the softmax
    denominator.  Rows are processed in blocks of one document so nothing
    N x N is formed.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    k_pos = np.asarray(k_pos, dtype=np.int64)
    nq, hq, d = q.shape
    nk, hkv, _ = k.shape
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    group = hq // hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((nq, hq, d))
    lse = np.full((hq, nq), -np.inf)
    if nq == 0 or nk == 0:
        return out, lse
    starts = doc_starts(cu_seqlens)
    q_start = starts[q_pos]
    k_order = np.argsort(k_pos, kind="stable")
    k_sorted = k_pos[k_order]
    for s, rows in _row_blocks(q_pos, q_start, row_block):
        last = q_pos[rows].max()
        lo = np.searchsorted(k_sorted, s, side="left")
        hi = np.searchsorted(k_sorted, last, side="right")
        keys = k_order[lo:hi]
        if keys.size == 0:
            continue
        # every key in [start, last] is in the document; causality is per row
        causal = k_pos[keys][None, :] <= q_pos[rows][:, None]
        for h in range(hq):
            g = h // group
            scores = (q[rows, h] @ k[keys, g].T) * scale
            scores = np.where(causal, scores, -np.inf)
            m = scores.max(axis=1)
            has_key = np.isfinite(m)
            m_safe = np.where(has_key, m, 0.0)
            p = np.exp(scores - m_safe[:, None])
            denom = p.sum(axis=1)
            o = (p @ v[keys, g]) / np.where(has_key, denom, 1.0)[:, None]
            out[rows, h] = np.where(has_key[:, None], o, 0.0)
            lse[h, rows] = np.where(has_key, m_safe + np.log(np.where(has_key, denom, 1.0)), -np.inf)
    return out, lse


def lse_merge(o_parts: List[np.ndarray], lse_parts: List[np.ndarray]):
    """Online-softmax combination of partial attention results.

    Each part p holds O_p [n, Hq, d] (normalised within its own key subset) and
    LSE_p [Hq, n].  With m = max_p LSE_p:
        L = m + ln sum_p exp(LSE_p - m),   O = sum_p exp(LSE_p - L) O_p.
    Rows where every part is -inf get O = 0 and L = -inf; a part whose LSE is
    -inf contributes nothing (its O rows are not read).
    """
    if not o_parts:
        raise ValueError("need at least one part")
    L = np.stack([_f64(x) for x in lse_parts])          # [p, Hq, n]
    m = L.max(axis=0)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    total = np.exp(L - m_safe[None]).sum(axis=0)
    lse = np.where(finite, m_safe + np.log(np.where(finite, total, 1.0)), -np.inf)
    out = np.zeros(_f64(o_parts[0]).shape)
    for o_p, l_p in zip(o_parts, L):
        present = np.isfinite(l_p)
        w = np.where(present, np.exp(np.where(present, l_p, 0.0) - np.where(finite, lse, 0.0)), 0.0)
        out += np.where(present.T[:, :, None], w.T[:, :, None] * _f64(o_p), 0.0)
    return out, lse


def attention_bwd(q, k, v, d_o, lse, delta, q_pos, k_pos, cu_seqlens,
                  scale: Optional[float] = None, row_block: int = 256):
    """Gradients of masked attention w.r.t. q, k, v for one set of key rows.

    ``lse`` [Hq, nq] is the log-sum-exp over ALL keys of each query row (the
    final, merged value) and ``delta`` [Hq, nq] = sum_d dO * O with the final
    O, so the probabilities P = exp(s - LSE) restricted to this key set are the
    entries of the full softmax.  From the definition:
        dV_j = sum_i P_ij dO_i,      dP_ij = dO_i . v_j,
        dS_ij = P_ij (dP_ij - delta_i),
        dQ_i = scale sum_j dS_ij k_j,   dK_j = scale sum_i dS_ij q_i,
    with dK, dV summed over the query heads that share a key/value head.
    Returns dq [nq, Hq, d], dk [nk, Hkv, d], dv [nk, Hkv, d].
    """
    q, k, v, d_o = _f64(q), _f64(k), _f64(v), _f64(d_o)
    lse, delta = _f64(lse), _f64(delta)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    k_pos = np.asarray(k_pos, dtype=np.int64)
    nq, hq, d = q.shape
    nk, hkv, _ = k.shape
    group = hq // hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    if nq == 0 or nk == 0:
        return dq, dk, dv
    starts = doc_starts(cu_seqlens)
    q_start = starts[q_pos]
    k_order = np.argsort(k_pos, kind="stable")
    k_sorted = k_pos[k_order]
    for s, rows in _row_blocks(q_pos, q_start, row_block):
        last = q_pos[rows].max()
        lo = np.searchsorted(k_sorted, s, side="left")
        hi = np.searchsorted(k_sorted, last, side="right")
        keys = k_order[lo:hi]
        if keys.size == 0:
            continue
        causal = k_pos[keys][None, :] <= q_pos[rows][:, None]
        for h in range(hq):
            g = h // group
            row_lse = lse[h, rows]
            ok = np.isfinite(row_lse)
            scores = (q[rows, h] @ k[keys, g].T) * scale
            with np.errstate(over="ignore", invalid="ignore"):
                p = np.where(causal & ok[:, None], np.exp(scores - np.where(ok, row_lse, 0.0)[:, None]), 0.0)
            dv[keys, g] += p.T @ d_o[rows, h]
            dp = d_o[rows, h] @ v[keys, g].T
            ds = p * (dp - delta[h, rows][:, None])
            dq[rows, h] += (ds @ k[keys, g]) * scale
            dk[keys, g] += (ds.T @ q[rows, h]) * scale
    return dq, dk, dv


def shard_forward(q, k, v, cu_seqlens, total_tokens: int, sp_degree: int, layout: str,
                  shard: int, scale: Optional[float] = None, rows: Optional[np.ndarray] = None) -> Dict:
    """Forward of one shard against every K/V chunk in ring order, then the merge.

    q, k, v are in global order ([N, Hq, d] and [N, Hkv, d]).  ``rows``
    optionally selects a subset of the shard's local query rows (for sampled
    checks at full size).  Returns a dict with
      ``chunks``   -- chunk id at each ring step,
      ``o_parts``/``lse_parts`` -- per ring step, partial O [n', Hq, d] and LSE [Hq, n'],
      ``o``/``lse`` -- merged result over all steps,
      ``q_pos``    -- global positions of the computed rows.
    """
    q_pos = shard_positions(total_tokens, sp_degree, layout, shard)
    if rows is not None:
        q_pos = q_pos[np.asarray(rows, dtype=np.int64)]
    qs = _f64(q[q_pos])
    chunks, o_parts, lse_parts = [], [], []
    for step in range(sp_degree):
        c = ring_chunk(shard, step, sp_degree)
        k_pos = shard_positions(total_tokens, sp_degree, layout, c)
        o_c, l_c = attention_fwd(qs, k[k_pos], v[k_pos], q_pos, k_pos, cu_seqlens, scale)
        chunks.append(c)
        o_parts.append(o_c)
        lse_parts.append(l_c)
    o, lse = lse_merge(o_parts, lse_parts)
    return {"chunks": chunks, "o_parts": o_parts, "lse_parts": lse_parts,
            "o": o, "lse": lse, "q_pos": q_pos}


def shard_backward(q, k, v, d_o, cu_seqlens, total_tokens: int, sp_degree: int, layout: str,
                   shard: int, scale: Optional[float] = None) -> Dict:
    """Backward of one shard: dQ for its rows and dK/dV contributions to every chunk.

    Recomputes the shard's forward (its own O and LSE) first; the
    probabilities of the backward come from that final LSE.  Returns
      ``dq``  [n, Hq, d] (shard-local row order),
      ``dk``/``dv`` [P, n, Hkv, d] indexed by chunk id, chunk-local row order,
      ``o``/``lse``/``delta`` of the forward, and ``fwd``, the forward's own dict.
    """
    fwd = shard_forward(q, k, v, cu_seqlens, total_tokens, sp_degree, layout, shard, scale)
    q_pos = fwd["q_pos"]
    qs = _f64(q[q_pos])
    dos = _f64(d_o[q_pos])
    delta = np.einsum("nhd,nhd->hn", dos, fwd["o"])
    n = len(q_pos)
    hkv, d = k.shape[1], k.shape[2]
    dq = np.zeros_like(qs)
    dk = np.zeros((sp_degree, n, hkv, d))
    dv = np.zeros((sp_degree, n, hkv, d))
    for c in range(sp_degree):
        k_pos = shard_positions(total_tokens, sp_degree, layout, c)
        dq_c, dk_c, dv_c = attention_bwd(qs, k[k_pos], v[k_pos], dos, fwd["lse"], delta,
                                         q_pos, k_pos, cu_seqlens, scale)
        dq += dq_c
        dk[c] = dk_c
        dv[c] = dv_c
    return {"dq": dq, "dk": dk, "dv": dv, "o": fwd["o"], "lse": fwd["lse"], "delta": delta, "fwd": fwd}
