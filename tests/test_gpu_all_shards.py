"""Every shard of a packed sequence on the GPU (ring and balanced schedules) against the fp64 oracle.

Bars as for the one-shard parity tests (O max-abs <= 2e-2, LSE max-abs <= 1e-3).
Both schedules compute every block with the same runs into the same partial
slots and merge each shard's parts in the same order, so their outputs must be
identical bit for bit; the balanced schedule must really move blocks where
the ring's loads are uneven (one causal document over contiguous shards).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from _harness import LSE_ATOL, O_ATOL, max_abs, oracle_by_kv_heads
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.all_shards import AllShards
from paper_2606_30460_amd.shard_attention import to_sharded
from workloads import make_workload, random_bf16

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _cu(rng, N, mean_len):
    lengths = []
    while sum(lengths) < N:
        lengths.append(int(rng.integers(1, 2 * mean_len)))
    lengths[-1] -= sum(lengths) - N
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


def _run(cu, N, P, layout, hq, hkv, d, bm, bn, seed, balance, max_run_tiles=None):
    q, k, v = random_bf16((N, hq, d), seed + 1), random_bf16((N, hkv, d), seed + 2), random_bf16((N, hkv, d), seed + 3)
    a = AllShards(cu, N, P, layout, hq, hkv, d, bm, bn, balance=balance, max_run_tiles=max_run_tiles)
    a.plan()
    dev = torch.device("cuda")
    s = L.shard_desc(N, P, layout, 0, bm, bn)
    q_sh, k_sh, v_sh = to_sharded(s, q.to(dev)), to_sharded(s, k.to(dev)), to_sharded(s, v.to(dev))
    bufs = a.alloc()
    bufs["o"].fill_(float("nan"))
    bufs["lse"].fill_(float("nan"))
    times = a.forward(q_sh, k_sh, v_sh, bufs, timed=True)
    torch.cuda.synchronize()
    return a, bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy(), times, (q, k, v)


CASES = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length (0: one document)
    (2048, 4, "contiguous", 4, 2, 128, 64, 64, 0),
    (2048, 4, "contiguous", 4, 2, 128, 128, 64, 300),
    (4096, 8, "zigzag", 4, 4, 64, 64, 64, 700),
    (4096, 8, "contiguous", 2, 1, 128, 64, 128, 1500),
    (4096, 2, "zigzag", 4, 2, 128, 256, 128, 0),
]


@pytest.mark.parametrize("case", CASES)
def test_all_shards_match_oracle_and_each_other(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    cu = np.array([0, N], dtype=np.int32) if mean == 0 else _cu(np.random.default_rng(N + P), N, mean)
    outs = {}
    for balance in (False, True):
        _say("all shards", case, "balanced" if balance else "ring")
        a, o, lse, times, (q, k, v) = _run(cu, N, P, layout, hq, hkv, d, bm, bn, seed=5, balance=balance)
        sched = a.schedule()
        _say(sched, {k_: [round(t, 3) for t in t_] for k_, t_ in times.items()})
        assert sum(sched["rank_tiles"]) == int(a.block_tiles.sum())
        outs[balance] = (o, lse)
        qf, kf, vf = q.float().numpy(), k.float().numpy(), v.float().numpy()
        for r in range(P):
            ref = oracle.shard_forward(qf, kf, vf, cu, N, P, layout, r)
            rep = {"o": max_abs(o[r], ref["o"]), "lse": max_abs(lse[r], ref["lse"])}
            assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, (r, rep)
        if balance and mean == 0 and layout == "contiguous":
            assert sched["moved_blocks"] > 0 and max(sched["rank_tiles"]) < int(a.block_tiles.sum(axis=1).max())
    assert np.array_equal(outs[False][0], outs[True][0]) and np.array_equal(outs[False][1], outs[True][1])


def test_all_shards_split_runs_agree():
    # shards whose long runs are split over several slots give the same bits whatever rank computes them
    N, P = 4096, 4
    cu = np.array([0, 3000, 3001, N], dtype=np.int32)
    res = [_run(cu, N, P, "contiguous", 4, 2, 128, 64, 64, seed=2, balance=b, max_run_tiles=3)[1:3] for b in (False, True)]
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])


def test_all_shards_workload_every_row():
    """The 32768-token log-normal workload, every shard (balanced schedule): every row against the
    oracle."""
    w = make_workload("c2")
    N, P = w.total_tokens, w.sp_degree
    a, o, lse, times, (q, k, v) = _run(w.cu_seqlens, N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim,
                                       w.block_m, w.block_n, seed=w.seed, balance=True)
    _say(a.schedule(), times)
    assert not np.isnan(o).any() and not np.isnan(lse).any()
    qf, kf, vf = q.float().numpy(), k.float().numpy(), v.float().numpy()
    for r in range(P):
        ref = oracle_by_kv_heads(qf, kf, vf, None, w.cu_seqlens, N, P, w.layout, r, list(range(w.heads_kv)))
        rep = {"o": max_abs(o[r], ref["o"]), "lse": max_abs(lse[r], ref["lse"])}
        _say("shard", r, rep)
        assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, (r, rep)
