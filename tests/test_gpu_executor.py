"""The step executor (hsap_executor_*) against the fp64 oracle and against the
per-entry-point path, on the same seeded inputs.

Bars as for the other parity tests (O max-abs <= 2e-2, LSE <= 1e-3, gradients
max|g - ref| / max|ref| <= 3e-2; the executor's gradients are bf16).  With the
same q-major split the executor launches the same kernels over the same lists
as the entry points called one by one, so O, LSE, the fused output and the
gradients (each block written by its one owning run, as bf16 directly or as
fp32 then converted) must be identical bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.plan import KIND_FULL, plan_shard
from _harness import GRAD_RTOL, LSE_ATOL, O_ATOL, Case, max_abs, rel_max
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.shard_attention import to_sharded

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


CASES = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length
    (1024, 1, "contiguous", 2, 2, 64, 64, 64, 300),
    (2048, 4, "zigzag", 4, 1, 128, 128, 64, 120),
    (4096, 4, "contiguous", 4, 2, 128, 128, 128, 1500),
    # documents of 1..5 tokens: up to 31 boundaries among a wave's 32 queries (the forwards find
    # document starts from cu_seqlens; the entry points read per-position starts)
    (2048, 2, "zigzag", 2, 2, 128, 256, 128, 3),
    (1024, 2, "contiguous", 2, 1, 64, 64, 64, 3),
]


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).float().numpy()


@pytest.mark.parametrize("case", CASES)
def test_executor_matches_oracle_and_entry_points(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    cu = _cu(np.random.default_rng(N + P), N, mean)
    r = P - 1
    bwd = True
    c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=20 + r, backward=bwd)
    ref = c.run_oracle()
    for split in (-1, 0, 1):
        _say("executor", case, "shard", r, "split", split)
        ex = c.run_executor(max_run_tiles=split)
        rep = {"o": max_abs(ex["o"], ref["fwd"]["o"]), "lse": max_abs(ex["lse"], ref["fwd"]["lse"]),
               "o_fused": max_abs(ex["o_fused"], ref["fwd"]["o"]), "lse_fused": max_abs(ex["lse_fused"], ref["fwd"]["lse"])}
        if bwd:
            rep.update(dq=rel_max(ex["dq"], ref["dq"]), dk=rel_max(ex["dk"], ref["dk"]), dv=rel_max(ex["dv"], ref["dv"]))
        _say(rep, ex["info"])
        assert rep["o"] <= O_ATOL and rep["o_fused"] <= O_ATOL, rep
        assert rep["lse"] <= LSE_ATOL and rep["lse_fused"] <= LSE_ATOL, rep
        if bwd:
            assert max(rep["dq"], rep["dk"], rep["dv"]) <= GRAD_RTOL, rep
        assert np.array_equal(ex["o_staged"], ex["o"]) and np.array_equal(ex["lse_staged"], ex["lse"])
        info = ex["info"]
        plan = plan_shard(cu, N, P, layout, r, bm, bn)
        assert info["num_tiles"] == len(plan["tiles"])
        assert info["num_full_tiles"] == int(np.sum(plan["tiles"][:, 3] == KIND_FULL))
        assert info["useful_pairs"] == int(plan["useful_pairs"].sum())
        if split >= 0:
            gpu = c.run_gpu(max_run_tiles=split)
            assert info["split_length"] == split
            assert info["num_parts"] == len(gpu["sa"].present)
            assert np.array_equal(ex["o"], gpu["o"]) and np.array_equal(ex["lse"], gpu["lse"])
            assert np.array_equal(ex["o_fused"], gpu["o_fused"]) and np.array_equal(ex["lse_fused"], gpu["lse_fused"])
            if bwd:
                assert np.array_equal(ex["dk"], _bf16(gpu["dk"])) and np.array_equal(ex["dv"], _bf16(gpu["dv"]))
                assert np.array_equal(ex["dq"], gpu["dq_bf16"])


# many (run, head) items, several times the GPU's resident workgroups, through the executor's
# partial and fused forwards and through the entry points
MANY_ITEMS = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length
    (8192, 2, "contiguous", 32, 32, 128, 128, 128, 300),
    # K/V heads a multiple of 8: a group's query heads placed on one XCD
    (16384, 4, "zigzag", 32, 8, 128, 128, 128, 500),
    # documents of 1..7 tokens: masked tiles throughout, runs of a single tile, chunks that no
    # query reaches
    (8192, 2, "contiguous", 32, 16, 128, 128, 128, 4),
    # one document: runs of up to 32 tiles (two windows), split into pieces by the planner
    (8192, 2, "contiguous", 32, 32, 128, 128, 128, 8192),
]


@pytest.mark.parametrize("case", MANY_ITEMS)
def test_executor_many_items(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    cu = _cu(np.random.default_rng(N + P + hkv), N, mean)
    r = P - 1
    c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=40 + r, backward=False)
    ref = c.run_oracle()
    for split in (-1, 0):
        _say("executor, many items", case, "shard", r, "split", split)
        ex = c.run_executor(max_run_tiles=split)
        info = ex["info"]
        assert info["num_runs_q"] * hq > 512 and info["num_runs_all"] * hq > 512, info
        rep = {"o": max_abs(ex["o"], ref["o"]), "lse": max_abs(ex["lse"], ref["lse"]),
               "o_fused": max_abs(ex["o_fused"], ref["o"]), "lse_fused": max_abs(ex["lse_fused"], ref["lse"])}
        _say(rep, info)
        assert rep["o"] <= O_ATOL and rep["o_fused"] <= O_ATOL, rep
        assert rep["lse"] <= LSE_ATOL and rep["lse_fused"] <= LSE_ATOL, rep
        assert np.array_equal(ex["o_staged"], ex["o"]) and np.array_equal(ex["lse_staged"], ex["lse"])
        gpu = c.run_gpu(max_run_tiles=info["split_length"])
        assert np.array_equal(ex["o"], gpu["o"]) and np.array_equal(ex["lse"], gpu["lse"])
        assert np.array_equal(ex["o_fused"], gpu["o_fused"]) and np.array_equal(ex["lse_fused"], gpu["lse_fused"])


def test_executor_replans_other_batches():
    """One executor, three batches in a row (the second needs more partials than the
    first, so the partial workspace grows), then the first batch again: every result
    meets the oracle, and the repeated batch gives the same bits."""
    N, P, layout, hq, hkv, d, bm, bn = 4096, 4, "contiguous", 4, 4, 128, 128, 128
    r = 2
    rng = np.random.default_rng(7)
    batches = [_cu(rng, N, 60),                                       # short documents: few partials
               np.array([0, N], dtype=np.int32),                     # one document: chunks 0..2, split in pieces
               _cu(rng, N, 2000)]
    s = L.shard_desc(N, P, layout, r, bm, bn)
    desc = L.attn_desc(s, hq, hkv, d, 1.0 / np.sqrt(d))
    ex = L.Executor(desc, backward=False, fused=True, max_run_tiles=1)
    dev = torch.device("cuda")
    c0 = Case(batches[0], N, P, layout, r, hq, hkv, d, bm, bn, seed=3)
    q_sh = to_sharded(s, c0.q.to(dev))[r].contiguous()
    k_sh, v_sh = to_sharded(s, c0.k.to(dev)), to_sharded(s, c0.v.to(dev))
    n = N // P
    results, parts = [], []
    try:
        for i, cu in enumerate(batches + [batches[0]]):
            _say("replan batch", i, "docs", len(cu) - 1)
            ex.plan(cu)
            o = torch.full((n, hq, d), float("nan"), dtype=torch.bfloat16, device=dev)
            lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device=dev)
            ex.forward(q_sh, k_sh, v_sh, o, lse)
            torch.cuda.synchronize()
            info = ex.info()
            parts.append(info["num_parts"])
            results.append((o.float().cpu().numpy(), lse.cpu().numpy()))
            ci = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=3)
            ref = ci.run_oracle()
            rep = {"o": max_abs(results[-1][0], ref["o"]), "lse": max_abs(results[-1][1], ref["lse"])}
            _say(info, rep)
            assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, rep
    finally:
        ex.close()
    assert parts[1] > parts[0]
    assert np.array_equal(results[0][0], results[3][0]) and np.array_equal(results[0][1], results[3][1])


def test_executor_many_plans_in_flight():
    """Forty plans of three different batches issued back to back with no synchronisation (the
    host runs ahead and reuses its pinned staging buffers while earlier uploads may still be in
    flight), each forward into its own outputs: every result equals, bit for bit, the first
    result of the same batch, and those meet the oracle."""
    N, P, layout, hq, hkv, d, bm, bn = 2048, 2, "contiguous", 2, 2, 128, 128, 128
    r = 1
    rng = np.random.default_rng(11)
    batches = [_cu(rng, N, 40), _cu(rng, N, 300), np.array([0, N], dtype=np.int32)]
    s = L.shard_desc(N, P, layout, r, bm, bn)
    desc = L.attn_desc(s, hq, hkv, d, 1.0 / np.sqrt(d))
    ex = L.Executor(desc, backward=False, fused=False, max_run_tiles=-1)
    dev = torch.device("cuda")
    c0 = Case(batches[0], N, P, layout, r, hq, hkv, d, bm, bn, seed=5)
    q_sh = to_sharded(s, c0.q.to(dev))[r].contiguous()
    k_sh, v_sh = to_sharded(s, c0.k.to(dev)), to_sharded(s, c0.v.to(dev))
    n = N // P
    outs = []
    try:
        for i in range(40):
            ex.plan(batches[i % 3])
            o = torch.full((n, hq, d), float("nan"), dtype=torch.bfloat16, device=dev)
            lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device=dev)
            ex.forward(q_sh, k_sh, v_sh, o, lse)
            outs.append((o, lse))
        torch.cuda.synchronize()
    finally:
        ex.close()
    got = [(o.float().cpu().numpy(), lse.cpu().numpy()) for o, lse in outs]
    for b in range(3):
        ref = Case(batches[b], N, P, layout, r, hq, hkv, d, bm, bn, seed=5).run_oracle()
        rep = {"o": max_abs(got[b][0], ref["o"]), "lse": max_abs(got[b][1], ref["lse"])}
        _say("batch", b, rep)
        assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, rep
        for i in range(b + 3, 40, 3):
            assert np.array_equal(got[i][0], got[b][0]) and np.array_equal(got[i][1], got[b][1]), (b, i)


def test_executor_rejects_misuse():
    s = L.shard_desc(2048, 2, "contiguous", 0, 128, 128)
    desc = L.attn_desc(s, 2, 2, 128, 0.1)
    ex = L.Executor(desc, backward=False, fused=False)
    dev = torch.device("cuda")
    try:
        q = torch.zeros(1024, 2, 128, dtype=torch.bfloat16, device=dev)
        kv = torch.zeros(2, 1024, 2, 128, dtype=torch.bfloat16, device=dev)
        o = torch.empty_like(q)
        lse = torch.empty(2, 1024, dtype=torch.float32, device=dev)
        with pytest.raises(L.HsapError):          # no plan yet
            ex.forward(q, kv, kv, o, lse)
        with pytest.raises(L.HsapError):
            ex.info()
        with pytest.raises(L.HsapError):          # cu_seqlens not ending at N
            ex.plan(np.array([0, 2000], dtype=np.int32))
        ex.plan(np.array([0, 2048], dtype=np.int32))
        with pytest.raises(L.HsapError):          # fused lists were not requested
            ex.forward(q, kv, kv, o, lse, fused=True)
        with pytest.raises(L.HsapError):          # no backward workspace
            ex.backward(q, kv, kv, q, o, lse, o, kv, kv)
        ex.forward(q, kv, kv, o, lse)
        torch.cuda.synchronize()
        # q = 0: every row averages V over its keys; V = 0 gives O = 0 and LSE = ln(i + 1)
        assert float(o.float().abs().max()) == 0.0
        ref = np.log(np.arange(1, 1025, dtype=np.float64))
        assert max_abs(lse.cpu().numpy()[0], ref) <= LSE_ATOL
    finally:
        ex.close()
