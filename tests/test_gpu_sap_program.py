"""The per-rank instruction lists executed on one GPU (one stream per rank) against the fp64 oracle.

Bars as for the other parity tests (O max-abs <= 2e-2, LSE max-abs <= 1e-3).  Every block is
computed by the same runs as in the all-shard execution without split, and each shard merges its
parts in chunk order, so the outputs must equal that execution's bit for bit, for the ring and the
balanced assignment alike.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from _harness import LSE_ATOL, O_ATOL, max_abs
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.all_shards import AllShards
from paper_2606_30460_amd.sap_program import SapProgram
from paper_2606_30460_amd.shard_attention import to_sharded
from workloads import make_workload, random_bf16

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _inputs(N, P, layout, hq, hkv, d, bm, bn, seed):
    q, k, v = random_bf16((N, hq, d), seed + 1), random_bf16((N, hkv, d), seed + 2), random_bf16((N, hkv, d), seed + 3)
    dev = torch.device("cuda")
    s = L.shard_desc(N, P, layout, 0, bm, bn)
    return (q, k, v), (to_sharded(s, q.to(dev)), to_sharded(s, k.to(dev)), to_sharded(s, v.to(dev)))


def _program(cu, N, P, layout, hq, hkv, d, bm, bn, balance, sharded):
    prog = SapProgram(cu, N, P, layout, hq, hkv, d, bm, bn, balance=balance)
    prog.plan()
    bufs = prog.alloc()
    bufs["o"].fill_(float("nan"))
    bufs["lse"].fill_(float("nan"))
    ms = prog.run(*sharded, bufs, timed=True)
    torch.cuda.synchronize()
    return prog, bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy(), ms


def _all_shards(cu, N, P, layout, hq, hkv, d, bm, bn, sharded):
    a = AllShards(cu, N, P, layout, hq, hkv, d, bm, bn, max_run_tiles=0)
    a.plan()
    bufs = a.alloc()
    a.forward(*sharded, bufs)
    torch.cuda.synchronize()
    return bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy()


CASES = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length (0: one document)
    (2048, 4, "contiguous", 4, 2, 128, 64, 64, 0),
    (4096, 8, "zigzag", 4, 4, 64, 64, 64, 700),
    (4096, 4, "contiguous", 2, 1, 128, 128, 128, 900),
    (4096, 2, "zigzag", 4, 2, 128, 256, 128, 0),
]


@pytest.mark.parametrize("case", CASES)
def test_program_matches_oracle_and_all_shards(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    rng = np.random.default_rng(N + 3 * P)
    if mean == 0:
        cu = np.array([0, N], dtype=np.int32)
    else:
        lengths = []
        while sum(lengths) < N:
            lengths.append(int(rng.integers(1, 2 * mean)))
        lengths[-1] -= sum(lengths) - N
        cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    (q, k, v), sharded = _inputs(N, P, layout, hq, hkv, d, bm, bn, seed=6)
    ref_bits = _all_shards(cu, N, P, layout, hq, hkv, d, bm, bn, sharded)
    qf, kf, vf = q.float().numpy(), k.float().numpy(), v.float().numpy()
    refs = [oracle.shard_forward(qf, kf, vf, cu, N, P, layout, r) for r in range(P)]
    for balance in (False, True):
        _say("program", case, "balanced" if balance else "ring")
        prog, o, lse, ms = _program(cu, N, P, layout, hq, hkv, d, bm, bn, balance, sharded)
        _say("stages", prog.num_stages, "ops", sum(len(x) for x in prog.ops), "ms", round(ms, 3))
        for r in range(P):
            rep = {"o": max_abs(o[r], refs[r]["o"]), "lse": max_abs(lse[r], refs[r]["lse"])}
            assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, (r, rep)
        assert np.array_equal(o, ref_bits[0]) and np.array_equal(lse, ref_bits[1])


def test_program_workload_bits():
    """The 32768-token log-normal workload: the balanced program gives the all-shard result bit for bit."""
    w = make_workload("c2")
    N, P = w.total_tokens, w.sp_degree
    _, sharded = _inputs(N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n, seed=w.seed)
    ref_bits = _all_shards(w.cu_seqlens, N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n,
                           sharded)
    prog, o, lse, ms = _program(w.cu_seqlens, N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m,
                                w.block_n, True, sharded)
    _say("c2 program: stages", prog.num_stages, "ms", round(ms, 3))
    assert np.array_equal(o, ref_bits[0]) and np.array_equal(lse, ref_bits[1])
