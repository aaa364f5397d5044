"""The per-rank instruction lists executed on one GPU (one stream per rank) against the fp64 oracle.

Bars as for the other parity tests (O max-abs <= 2e-2, LSE max-abs <= 1e-3, gradients
max|g - ref| / max|ref| <= 3e-2).  The backward program's gradients (every block's parts summed
in part order) must equal the all-shard backward's bit for bit, for the ring and the balanced
assignment alike.  Every block is
computed by the same runs as in the all-shard execution without split, and each shard merges its
parts in chunk order, so the outputs must equal that execution's bit for bit, for the ring and the
balanced assignment alike.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from _harness import GRAD_RTOL, LSE_ATOL, O_ATOL, max_abs, oracle_by_kv_heads, rel_max
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


# ---------------------------------------------------------------------------
# backward program (hsap_emit_backward): dq, dkv and do messages
# ---------------------------------------------------------------------------

def _backward_inputs(N, P, layout, hq, hkv, d, bm, bn, seed):
    (q, k, v), sharded = _inputs(N, P, layout, hq, hkv, d, bm, bn, seed)
    do = random_bf16((N, hq, d), seed + 4)
    s = L.shard_desc(N, P, layout, 0, bm, bn)
    return (q, k, v, do), sharded + (to_sharded(s, do.to(torch.device("cuda"))),)


def _forward_outputs(cu, N, P, layout, hq, hkv, d, bm, bn, sharded):
    a = AllShards(cu, N, P, layout, hq, hkv, d, bm, bn, max_run_tiles=0)
    a.plan()
    bufs = a.alloc()
    a.forward(*sharded[:3], bufs)
    return bufs["o"], bufs["lse"]


def _all_shards_backward(cu, N, P, layout, hq, hkv, d, bm, bn, sharded, o, lse, balance):
    a = AllShards(cu, N, P, layout, hq, hkv, d, bm, bn, balance=balance, max_run_tiles=0)
    a.plan(backward=True)
    bufs = a.alloc_backward()
    for key in ("dq", "dk", "dv"):
        bufs[key].fill_(float("nan"))
    q, k, v, do = sharded
    times = a.backward(q, k, v, do, o, lse, bufs, timed=True)
    torch.cuda.synchronize()
    return [bufs[x].float().cpu().numpy() for x in ("dq", "dk", "dv")], times


def _program_backward(cu, N, P, layout, hq, hkv, d, bm, bn, sharded, o, lse, balance):
    prog = SapProgram(cu, N, P, layout, hq, hkv, d, bm, bn, balance=balance)
    prog.plan(backward=True)
    bufs = prog.alloc_backward()
    for key in ("dq", "dk", "dv"):
        bufs[key].fill_(float("nan"))
    q, k, v, do = sharded
    ms = prog.run_backward(q, k, v, do, o, lse, bufs, timed=True)
    torch.cuda.synchronize()
    return prog, [bufs[x].float().cpu().numpy() for x in ("dq", "dk", "dv")], ms


def _oracle_gradients(cu, N, P, layout, host, kv_heads=None):
    """dQ of every shard and dK/dV of every chunk summed over the shards' contributions (fp64)."""
    q, k, v, do = (t.float().numpy() for t in host)
    kv = list(range(k.shape[1])) if kv_heads is None else kv_heads
    dq, dk, dv = [], 0.0, 0.0
    for r in range(P):
        g = oracle_by_kv_heads(q, k, v, do, cu, N, P, layout, r, kv)
        dq.append(g["dq"])
        dk = dk + g["dk"]
        dv = dv + g["dv"]
    return np.stack(dq), dk, dv


BWD_CASES = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length (0: one document)
    (2048, 4, "contiguous", 4, 2, 128, 64, 64, 0),
    (4096, 8, "zigzag", 4, 4, 64, 64, 64, 700),
    (4096, 4, "contiguous", 2, 1, 128, 128, 128, 900),
    (4096, 2, "zigzag", 4, 2, 128, 256, 128, 0),
]


@pytest.mark.parametrize("case", BWD_CASES)
def test_backward_program_matches_oracle_and_all_shards(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    rng = np.random.default_rng(N + 5 * P)
    if mean == 0:
        cu = np.array([0, N], dtype=np.int32)
    else:
        lengths = []
        while sum(lengths) < N:
            lengths.append(int(rng.integers(1, 2 * mean)))
        lengths[-1] -= sum(lengths) - N
        cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    host, sharded = _backward_inputs(N, P, layout, hq, hkv, d, bm, bn, seed=8)
    o, lse = _forward_outputs(cu, N, P, layout, hq, hkv, d, bm, bn, sharded)
    ref_bits, times = _all_shards_backward(cu, N, P, layout, hq, hkv, d, bm, bn, sharded, o, lse, False)
    _say("all-shard backward", case, {k_: [round(t, 3) for t in t_] for k_, t_ in times.items()})
    for x in ref_bits:
        assert not np.isnan(x).any()
    dq_ref, dk_ref, dv_ref = _oracle_gradients(cu, N, P, layout, host)
    rep = {"dq": rel_max(ref_bits[0], dq_ref), "dk": rel_max(ref_bits[1], dk_ref), "dv": rel_max(ref_bits[2], dv_ref)}
    _say("vs oracle", rep)
    assert max(rep.values()) <= GRAD_RTOL, rep
    bal_bits, _ = _all_shards_backward(cu, N, P, layout, hq, hkv, d, bm, bn, sharded, o, lse, True)
    assert all(np.array_equal(a, b) for a, b in zip(bal_bits, ref_bits))
    for balance in (False, True):
        prog, bits, ms = _program_backward(cu, N, P, layout, hq, hkv, d, bm, bn, sharded, o, lse, balance)
        _say("backward program", "balanced" if balance else "ring", "stages", prog.num_stages_bwd, "ops",
             sum(len(x) for x in prog.ops_bwd), "ms", round(ms, 3))
        assert all(np.array_equal(a, b) for a, b in zip(bits, ref_bits)), balance


def test_backward_program_workload():
    """The 32768-token log-normal workload, forward + backward, balanced program: the all-shard
    backward's bits, and the oracle on two K/V heads."""
    w = make_workload("c2")
    N, P = w.total_tokens, w.sp_degree
    args = (w.cu_seqlens, N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n)
    host, sharded = _backward_inputs(N, P, w.layout, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n,
                                     seed=w.seed)
    o, lse = _forward_outputs(*args, sharded)
    ref_bits, times = _all_shards_backward(*args, sharded, o, lse, False)
    prog, bits, ms = _program_backward(*args, sharded, o, lse, True)
    _say("c2 backward program: stages", prog.num_stages_bwd, "ms", round(ms, 3), "all-shard ranks", times)
    assert all(np.array_equal(a, b) for a, b in zip(bits, ref_bits))
    kv = [0, w.heads_kv - 1]
    dq_ref, dk_ref, dv_ref = _oracle_gradients(w.cu_seqlens, N, P, w.layout, host, kv)
    hs = np.concatenate([np.arange(g * (w.heads_q // w.heads_kv), (g + 1) * (w.heads_q // w.heads_kv)) for g in kv])
    rep = {"dq": rel_max(bits[0][:, :, hs], dq_ref), "dk": rel_max(bits[1][:, :, kv], dk_ref),
           "dv": rel_max(bits[2][:, :, kv], dv_ref)}
    _say("c2 vs oracle on K/V heads", kv, rep)
    assert max(rep.values()) <= GRAD_RTOL, rep
