"""Batches of packed sequences through the step executor against the batched fp64 oracle.

Bars as for the single-sequence parity tests: O max-abs <= 2e-2, LSE max-abs <= 1e-3,
gradients max|g - ref| / max|ref| <= 3e-2.  The batch's rows are b*n + l for every shard and
chunk; attention never crosses a sequence, so each sequence's rows must match that sequence's
own oracle result.  A batch of copies of one sequence must give the copies of its result bit for
bit (the same tiles and runs, shifted).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from _harness import GRAD_RTOL, LSE_ATOL, O_ATOL, max_abs, oracle_by_kv_heads, rel_max
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.shard_attention import to_sharded
from workloads import make_workload, random_bf16

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _seq_cu(rng, N, mean_len):
    lengths = []
    while sum(lengths) < N:
        lengths.append(int(rng.integers(1, 2 * mean_len)))
    lengths[-1] -= sum(lengths) - N
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)


def _batch_cu(cus, N):
    return np.concatenate([cus[0]] + [c[1:] + b * N for b, c in enumerate(cus) if b > 0]).astype(np.int32)


def _run(cu, N, B, P, layout, r, hq, hkv, d, bm, bn, tensors, backward, split=-1):
    s = L.shard_desc(N, P, layout, r, bm, bn, batch=B)
    desc = L.attn_desc(s, hq, hkv, d, 1.0 / float(np.sqrt(d)))
    ex = L.Executor(desc, backward=backward, fused=True, max_run_tiles=split)
    dev = torch.device("cuda")
    q, k, v = (to_sharded(s, tensors[x].to(dev)) for x in ("q", "k", "v"))
    q = q[r].contiguous()
    n = s.rows
    out = {}
    try:
        ex.plan(cu)
        o = torch.full((n, hq, d), float("nan"), dtype=torch.bfloat16, device=dev)
        lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device=dev)
        ex.forward(q, k, v, o, lse)
        of, lf = torch.full_like(o, float("nan")), torch.full_like(lse, float("nan"))
        ex.forward(q, k, v, of, lf, fused=True)
        out.update(o=o.float().cpu().numpy(), lse=lse.cpu().numpy(), o_fused=of.float().cpu().numpy(),
                   lse_fused=lf.cpu().numpy(), info=ex.info())
        if backward:
            do = to_sharded(s, tensors["do"].to(dev))[r].contiguous()
            dq = torch.full_like(q, float("nan"))
            dk, dv = torch.zeros_like(k), torch.zeros_like(v)
            ex.backward(q, k, v, do, o, lse, dq, dk, dv)
            out.update(dq=dq.float().cpu().numpy(), dk=dk.float().cpu().numpy(), dv=dv.float().cpu().numpy())
        torch.cuda.synchronize()
    finally:
        ex.close()
    return out


CASES = [
    # N per sequence, B, P, layout, hq, hkv, d, bm, bn, mean doc length, backward
    (1024, 3, 2, "contiguous", 4, 2, 128, 64, 64, 200, True),
    (2048, 2, 4, "zigzag", 4, 4, 64, 64, 64, 300, True),
    (2048, 4, 4, "contiguous", 2, 1, 128, 128, 128, 700, True),
    (4096, 2, 2, "zigzag", 4, 2, 128, 256, 128, 1500, True),
]


@pytest.mark.parametrize("case", CASES)
def test_batch_matches_oracle(case):
    N, B, P, layout, hq, hkv, d, bm, bn, mean, bwd = case
    rng = np.random.default_rng(N + B * 10 + P)
    cu = _batch_cu([_seq_cu(rng, N, mean) for _ in range(B)], N)
    tensors = {"q": random_bf16((B * N, hq, d), 11), "k": random_bf16((B * N, hkv, d), 12),
               "v": random_bf16((B * N, hkv, d), 13)}
    if bwd:
        tensors["do"] = random_bf16((B * N, hq, d), 14)
    f = {x: t.float().numpy() for x, t in tensors.items()}
    for r in sorted({0, P - 1}):
        _say("batch", case, "shard", r)
        got = _run(cu, N, B, P, layout, r, hq, hkv, d, bm, bn, tensors, bwd)
        ref = oracle.batch_shard_forward(f["q"], f["k"], f["v"], cu, N, B, P, layout, r)
        rep = {"o": max_abs(got["o"], ref["o"]), "lse": max_abs(got["lse"], ref["lse"]),
               "o_fused": max_abs(got["o_fused"], ref["o"]), "lse_fused": max_abs(got["lse_fused"], ref["lse"])}
        if bwd:
            g = oracle.batch_shard_backward(f["q"], f["k"], f["v"], f["do"], cu, N, B, P, layout, r)
            rep.update(dq=rel_max(got["dq"], g["dq"]), dk=rel_max(got["dk"], g["dk"]), dv=rel_max(got["dv"], g["dv"]))
        _say(rep, got["info"])
        assert max(rep["o"], rep["o_fused"]) <= O_ATOL and max(rep["lse"], rep["lse_fused"]) <= LSE_ATOL, rep
        if bwd:
            assert max(rep["dq"], rep["dk"], rep["dv"]) <= GRAD_RTOL, rep


def test_batch_of_copies_gives_copies():
    N, B, P, layout, hq, d = 2048, 3, 4, "zigzag", 4, 128
    seq = _seq_cu(np.random.default_rng(5), N, 400)
    cu = _batch_cu([seq] * B, N)
    one = {x: random_bf16((N, hq, d), 20 + i) for i, x in enumerate(("q", "k", "v"))}
    tensors = {x: torch.cat([t] * B) for x, t in one.items()}
    n = N // P
    for r in range(P):
        got = _run(cu, N, B, P, layout, r, hq, hq, d, 64, 64, tensors, False, split=0)
        for b in range(1, B):
            assert np.array_equal(got["o"][b * n:(b + 1) * n], got["o"][:n])
            assert np.array_equal(got["lse"][:, b * n:(b + 1) * n], got["lse"][:, :n])


def test_batch_workload_every_row():
    """Four 32768-token log-normal sequences in one call (the batched workload), every row of every
    sequence against the oracle run on that sequence alone."""
    w = make_workload("c6")
    N, B, P, r = w.total_tokens, w.batch, w.sp_degree, w.shard
    tensors = w.tensors(backward=False)
    got = _run(w.cu_seqlens, N, B, P, w.layout, r, w.heads_q, w.heads_kv, w.head_dim, w.block_m, w.block_n,
               tensors, False)
    f = {x: t.float().numpy() for x, t in tensors.items()}
    n = N // P
    for key in ("o", "lse", "o_fused", "lse_fused"):
        assert not np.isnan(got[key]).any(), key
    for b, cu_b in enumerate(oracle.split_batch(w.cu_seqlens, N, B)):
        sl = slice(b * N, (b + 1) * N)
        ref = oracle_by_kv_heads(f["q"][sl], f["k"][sl], f["v"][sl], None, cu_b, N, P, w.layout, r,
                                 list(range(w.heads_kv)))
        rows = slice(b * n, (b + 1) * n)
        rep = {"o": max_abs(got["o"][rows], ref["o"]), "lse": max_abs(got["lse"][:, rows], ref["lse"]),
               "o_fused": max_abs(got["o_fused"][rows], ref["o"]),
               "lse_fused": max_abs(got["lse_fused"][:, rows], ref["lse"])}
        _say("sequence", b, rep)
        assert max(rep["o"], rep["o_fused"]) <= O_ATOL and max(rep["lse"], rep["lse_fused"]) <= LSE_ATOL, (b, rep)
