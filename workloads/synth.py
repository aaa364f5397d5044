"""Document-length samplers, packed-sequence workloads and seeded bf16 tensors.

Seeding convention (base seed ``s``, default 0):
  * document lengths: ``numpy.random.default_rng(s)``;
  * Q, K, V, dO: ``torch.Generator().manual_seed(s + 1 .. s + 4)``, drawn as
    N(0, 1) float32 and rounded to bfloat16 (round-to-nearest-even, torch's
    conversion).

Every sampler returns a Python list of positive ints summing to the requested
total.  ``cu_seqlens_from_lengths`` turns lengths into the cumulative-length
array that the packed-attention interface takes (first entry 0, last entry the
total token count).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional

import numpy as np
import torch


# ---------------------------------------------------------------------------
# document-length samplers
# ---------------------------------------------------------------------------

def doc_lengths_uniform_partition(total: int, num_docs: int, min_len: int, seed: int = 0) -> List[int]:
    """Uniform random composition of ``total`` into ``num_docs`` parts, each >= ``min_len``.

    ``num_docs - 1`` cut points are drawn iid uniformly from the inclusive range
    ``0 .. total - num_docs*min_len`` and sorted; the gaps plus ``min_len`` are
    the lengths.
    """
    free = total - num_docs * min_len
    if free < 0:
        raise ValueError("total too small for num_docs * min_len")
    rng = np.random.default_rng(seed)
    cuts = np.sort(rng.integers(0, free, size=num_docs - 1, endpoint=True))
    gaps = np.diff(np.concatenate([[0], cuts, [free]]))
    return [int(g) + min_len for g in gaps]


def _truncate_to_total(lengths: List[int], total: int) -> List[int]:
    out: List[int] = []
    acc = 0
    for length in lengths:
        if acc >= total:
            break
        take = min(length, total - acc)
        if take > 0:
            out.append(int(take))
            acc += take
    if acc != total:
        raise ValueError("lengths do not cover total")
    return out


def doc_lengths_lognormal(total: int, median: float, sigma: float, lo: int, hi: int,
                          seed: int = 0) -> List[int]:
    """Log-normal lengths (natural-log sigma), rounded, clamped to [lo, hi].

    Draws until the running sum reaches ``total``; the last document is cut so
    the lengths sum to ``total`` exactly.
    """
    rng = np.random.default_rng(seed)
    mu = math.log(median)
    lengths: List[int] = []
    acc = 0
    while acc < total:
        x = int(round(float(rng.lognormal(mean=mu, sigma=sigma))))
        x = min(max(x, lo), hi)
        lengths.append(x)
        acc += x
    return _truncate_to_total(lengths, total)


def doc_lengths_mixed(total: int, p_long: float, short: tuple, long: tuple, seed: int = 0) -> List[int]:
    """Two-population mixture: with probability ``p_long`` a length uniform in
    ``long`` (inclusive), else uniform in ``short`` (inclusive).

    Draws until the sum reaches ``total``, shuffles the drawn list with the same
    generator, then keeps documents in shuffled order until ``total`` tokens are
    covered (the last kept one cut to fit, the rest dropped).
    """
    rng = np.random.default_rng(seed)
    lengths: List[int] = []
    acc = 0
    while acc < total:
        if rng.random() < p_long:
            x = int(rng.integers(long[0], long[1], endpoint=True))
        else:
            x = int(rng.integers(short[0], short[1], endpoint=True))
        lengths.append(x)
        acc += x
    order = rng.permutation(len(lengths))
    return _truncate_to_total([lengths[i] for i in order], total)


def doc_lengths_pareto(total: int, alpha: float, xmin: int, xmax: int, seed: int = 0) -> List[int]:
    """Classic Pareto lengths ``floor(xmin * (1 + Lomax(alpha)))`` clamped at ``xmax``.

    numpy's ``pareto`` draws the Lomax (Pareto II) variate, hence the ``1 +``.
    """
    rng = np.random.default_rng(seed)
    lengths: List[int] = []
    acc = 0
    while acc < total:
        x = int(math.floor(xmin * (1.0 + float(rng.pareto(alpha)))))
        x = min(max(x, xmin), xmax)
        lengths.append(x)
        acc += x
    return _truncate_to_total(lengths, total)


def doc_lengths_extreme(total: int, long_len: int, short_len: int, long_first: bool = True) -> List[int]:
    """One long document plus short documents filling the rest of ``total``."""
    rest = total - long_len
    if rest < 0 or rest % short_len != 0:
        raise ValueError("remaining tokens must be a multiple of short_len")
    shorts = [short_len] * (rest // short_len)
    return [long_len] + shorts if long_first else shorts + [long_len]


def cu_seqlens_from_lengths(lengths: List[int]) -> np.ndarray:
    """Cumulative lengths as int32 ``[len(lengths) + 1]`` starting at 0."""
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    if cu[-1] > np.iinfo(np.int32).max:
        raise ValueError("total tokens exceed int32")
    return cu.astype(np.int32)


# ---------------------------------------------------------------------------
# tensors
# ---------------------------------------------------------------------------

def random_bf16(shape, seed: int) -> torch.Tensor:
    """N(0, 1) float32 draws from a seeded CPU generator, rounded to bfloat16."""
    g = torch.Generator().manual_seed(int(seed))
    return torch.randn(*shape, generator=g, dtype=torch.float32).to(torch.bfloat16)


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Workload:
    """One packed-sequence attention problem for a single sequence-parallel shard.

    ``shard`` is the shard id, or ``None`` meaning "the shard with the most
    useful (unmasked) query-key pairs" -- the slowest rank, which sets the step
    time of a sequence-parallel group.  Picking it needs the mask, so the
    caller resolves it with its own planner.

    ``batch`` packed sequences of ``total_tokens`` tokens each are concatenated
    (``lengths`` lists every sequence's documents in turn, each sequence's
    summing to ``total_tokens``); tensors then have batch * total_tokens rows.
    """
    name: str
    total_tokens: int
    lengths: List[int]
    heads_q: int
    heads_kv: int
    head_dim: int
    sp_degree: int
    layout: str              # "contiguous" or "zigzag"
    shard: Optional[int]
    block_m: int
    block_n: int
    backward: bool
    seed: int = 0
    batch: int = 1

    @property
    def cu_seqlens(self) -> np.ndarray:
        return cu_seqlens_from_lengths(self.lengths)

    @property
    def num_docs(self) -> int:
        return len(self.lengths)

    def tensors(self, backward: Optional[bool] = None) -> Dict[str, torch.Tensor]:
        """Q [B*N, Hq, d], K and V [B*N, Hkv, d] (and dO [B*N, Hq, d]) in global token order."""
        bwd = self.backward if backward is None else backward
        N, hq, hkv, d = self.total_tokens * self.batch, self.heads_q, self.heads_kv, self.head_dim
        out = {
            "q": random_bf16((N, hq, d), self.seed + 1),
            "k": random_bf16((N, hkv, d), self.seed + 2),
            "v": random_bf16((N, hkv, d), self.seed + 3),
        }
        if bwd:
            out["do"] = random_bf16((N, hq, d), self.seed + 4)
        return out


def _c1(seed: int) -> Workload:
    return Workload("c1_n2048_6docs_h4_d64_sp1", 2048,
                    doc_lengths_uniform_partition(2048, 6, 16, seed), 4, 4, 64,
                    1, "contiguous", 0, 64, 64, False, seed)


def _c2(seed: int) -> Workload:
    return Workload("c2_n32k_lognormal_h32_d128_sp8_shard3", 32768,
                    doc_lengths_lognormal(32768, 2048.0, 1.0, 128, 16384, seed), 32, 32, 128,
                    8, "contiguous", 3, 128, 128, False, seed)


def _c3(seed: int) -> Workload:
    return Workload("c3_n128k_mixed_gqa32x8_d128_sp16_zigzag", 131072,
                    doc_lengths_mixed(131072, 0.1, (64, 512), (8192, 65536), seed), 32, 8, 128,
                    16, "zigzag", None, 128, 128, False, seed)


def _c4(seed: int) -> Workload:
    return Workload("c4_n256k_pareto_h8of32_d128_ring8", 262144,
                    doc_lengths_pareto(262144, 1.2, 32, 131072, seed), 8, 8, 128,
                    8, "contiguous", None, 128, 128, False, seed)


def _c5(seed: int) -> Workload:
    return Workload("c5_n32k_30000plus346x8_h32_d128_sp8_shard0_fwdbwd", 32768,
                    doc_lengths_extreme(32768, 30000, 8, long_first=True), 32, 32, 128,
                    8, "contiguous", 0, 128, 128, True, seed)


def _c5m(seed: int) -> Workload:
    return Workload("c5m_n32k_346x8plus30000_h32_d128_sp8_shard0_fwdbwd", 32768,
                    doc_lengths_extreme(32768, 30000, 8, long_first=False), 32, 32, 128,
                    8, "contiguous", 0, 128, 128, True, seed)


def _c6(seed: int) -> Workload:
    # four packed sequences of the log-normal mix (each with its own documents) in one call
    lengths: List[int] = []
    for b in range(4):
        lengths += doc_lengths_lognormal(32768, 2048.0, 1.0, 128, 16384, seed + 1000 * b)
    return Workload("c6_4x32k_lognormal_h32_d128_sp8_shard3", 32768, lengths, 32, 32, 128,
                    8, "contiguous", 3, 128, 128, False, seed, batch=4)


CONFIGS: Dict[str, Callable[[int], Workload]] = {
    "c1": _c1, "c2": _c2, "c3": _c3, "c4": _c4, "c5": _c5, "c5m": _c5m, "c6": _c6,
}


def make_workload(name: str, seed: int = 0) -> Workload:
    return CONFIGS[name](seed)
