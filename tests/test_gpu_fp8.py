"""The fp8 score variant on the GPU: e4m3 quantisation bit for bit against the oracle, and the
fp8 partial forward (plus the merge) against the oracle's attention on the dequantised Q and K.

Bars: codes and scales identical (integer work); O max-abs <= 2e-2, LSE max-abs <= 1e-3 and the
-inf rows of every partial identical, as for the bf16 path -- the reference is the attention of
exactly the values the fp8 operands encode, so only accumulation order differs.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from _harness import LSE_ATOL, O_ATOL, max_abs, oracle_by_kv_heads
from paper_2606_30460_amd import _lib as L
from paper_2606_30460_amd.shard_attention import ShardAttention, to_sharded
from workloads import make_workload, random_bf16

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _quantize(x):
    codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    scale = torch.empty(x.shape[0], x.shape[2], dtype=torch.float32, device=x.device)
    work = torch.full((x.shape[0] * x.shape[2] * L.QUANT_SPLIT,), float("nan"), dtype=torch.float32, device=x.device)
    L.quantize_fp8(x, codes, scale, work)
    return codes, scale


@pytest.mark.parametrize("shape", [(1, 4096, 32, 128), (8, 256, 4, 128), (3, 100, 2, 64), (2, 1, 1, 8)])
def test_quantize_bit_exact(shape):
    G, rows, H, d = shape
    g = torch.Generator().manual_seed(G * rows + H)
    x = torch.randn(shape, generator=g) * torch.logspace(-3, 2, H).view(1, 1, H, 1)
    x = x.to(torch.bfloat16)
    if G > 1:
        x[1, :, 0, :] = 0          # a slice with amax 0
    codes, scale = _quantize(x.cuda())
    torch.cuda.synchronize()
    ref_codes, ref_scale = oracle.quantize_fp8(x.float().numpy())
    assert np.array_equal(codes.cpu().numpy(), ref_codes)
    assert np.array_equal(scale.cpu().numpy(), ref_scale)


def _fp8_forward(cu, N, P, layout, r, hq, hkv, d, bm, bn, q, k, v, split=None):
    """Plan shard r, quantise its Q and every chunk's K on the GPU, run the fp8 partial forward and
    the merge.  Returns GPU outputs and the oracle's dequantised Q / K in global order: the
    oracle quantises the same bf16 inputs itself (its codes and scales must equal the GPU's bit
    for bit), so no oracle input comes from the GPU."""
    sa = ShardAttention(cu, N, P, layout, r, hq, hkv, d, bm, bn, max_run_tiles=split)
    sa.plan()
    dev = torch.device("cuda")
    s = sa.shard
    q_sh = to_sharded(s, q.to(dev))[r].contiguous()
    k_sh, v_sh = to_sharded(s, k.to(dev)), to_sharded(s, v.to(dev))
    q8, qs = _quantize(q_sh.unsqueeze(0))
    k8, ks = _quantize(k_sh)
    bufs = sa.alloc_forward()
    bufs["lse_part"].fill_(float("nan"))
    L.partial_attn_fwd_fp8(sa.desc, q8, k8, v_sh, qs, ks, sa.doc_start, sa.tiles_q, sa.runs_q, bufs["o_part"],
                           bufs["lse_part"])
    L.lse_merge([bufs["o_part"][x] for x in sa.present], [bufs["lse_part"][x] for x in sa.present], sa.n, hq, d,
                bufs["o"], bufs["lse"])
    torch.cuda.synchronize()
    # the oracle's own quantisation of shard r's Q and of every chunk's K (sharded order, as
    # the codes are laid out), dequantised back into global order
    qf, kf = q.float().numpy(), k.float().numpy()
    q_pos = oracle.shard_positions(N, P, layout, r)
    k_sh = np.stack([kf[oracle.shard_positions(N, P, layout, c)] for c in range(P)])
    rq8, rqs = oracle.quantize_fp8(qf[q_pos][None])
    rk8, rks = oracle.quantize_fp8(k_sh)
    assert np.array_equal(q8.cpu().numpy(), rq8) and np.array_equal(qs.cpu().numpy(), rqs)
    assert np.array_equal(k8.cpu().numpy(), rk8) and np.array_equal(ks.cpu().numpy(), rks)
    q_deq = np.zeros((N, hq, d))
    k_deq = np.zeros((N, hkv, d))
    q_deq[q_pos] = oracle.dequantize_fp8(rq8, rqs)[0]
    kd = oracle.dequantize_fp8(rk8, rks)
    for c in range(P):
        k_deq[oracle.shard_positions(N, P, layout, c)] = kd[c]
    return sa, bufs, q_deq, k_deq


def _cu(rng, N, mean_len):
    lengths = []
    while sum(lengths) < N:
        lengths.append(int(rng.integers(1, 2 * mean_len)))
    lengths[-1] -= sum(lengths) - N
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


CASES = [
    # N, P, layout, hq, hkv, bm, bn, mean doc length
    (2048, 2, "contiguous", 4, 2, 128, 128, 300),
    (2048, 4, "zigzag", 4, 4, 64, 64, 150),
    (4096, 4, "contiguous", 2, 1, 128, 64, 900),
    (4096, 2, "zigzag", 4, 2, 256, 128, 700),
]


@pytest.mark.parametrize("case", CASES)
def test_fp8_forward_matches_oracle(case):
    N, P, layout, hq, hkv, bm, bn, mean = case
    d = 128
    cu = _cu(np.random.default_rng(N + P), N, mean)
    q, k, v = random_bf16((N, hq, d), 31), random_bf16((N, hkv, d), 32), random_bf16((N, hkv, d), 33)
    for r in sorted({0, P - 1}):
        _say("fp8 forward", case, "shard", r)
        sa, bufs, q_deq, k_deq = _fp8_forward(cu, N, P, layout, r, hq, hkv, d, bm, bn, q, k, v)
        ref = oracle.shard_forward(q_deq, k_deq, v.float().numpy(), cu, N, P, layout, r)
        o, lse = bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy()
        lse_part = bufs["lse_part"].cpu().numpy()
        rep = {"o": max_abs(o, ref["o"]), "lse": max_abs(lse, ref["lse"])}
        for step, c in enumerate(ref["chunks"]):
            slots = [x for x in sa.present if x % P == c]
            if len(slots) == 1:
                assert np.array_equal(np.isneginf(lse_part[slots[0]]), np.isneginf(ref["lse_parts"][step]))
        _say(rep)
        assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, rep


def test_fp8_forward_workload_every_row():
    """The 32768-token log-normal workload's shard with fp8 scores: every row against the oracle."""
    w = make_workload("c2")
    t = w.tensors(backward=False)
    sa, bufs, q_deq, k_deq = _fp8_forward(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, w.shard, w.heads_q,
                                          w.heads_kv, w.head_dim, w.block_m, w.block_n, t["q"], t["k"], t["v"])
    ref = oracle_by_kv_heads(q_deq, k_deq, t["v"].float().numpy(), None, w.cu_seqlens, w.total_tokens, w.sp_degree,
                             w.layout, w.shard, list(range(w.heads_kv)))
    o, lse = bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy()
    assert not np.isnan(o).any() and not np.isnan(lse).any()
    rep = {"o": max_abs(o, ref["o"]), "lse": max_abs(lse, ref["lse"])}
    _say(rep)
    assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, rep


@pytest.mark.parametrize("bm", [128, 64])
def test_fp8_forward_zero_slices(bm):
    """A K chunk that is all zeros and a query head that is all zeros quantise with scale 0: their
    scores are all 0, so those rows attend uniformly over their allowed keys (the oracle's
    result), never NaN from a masked score times a zero scale (direct-to-LDS kernel at 128-row
    q-tiles, register-staged kernel at 64)."""
    N, P, layout, hq, hkv, d, bn = 2048, 4, "contiguous", 4, 2, 128, 64
    cu = np.array([0, 300, 301, 900, 1500, 2048], dtype=np.int32)
    q, k, v = random_bf16((N, hq, d), 41), random_bf16((N, hkv, d), 42), random_bf16((N, hkv, d), 43)
    q[:, 1] = 0                                                   # query head 1: amax 0 on every shard
    k[oracle.shard_positions(N, P, layout, 1)] = 0                # chunk 1: amax 0 for both K/V heads
    for r in (1, 2, 3):
        sa, bufs, q_deq, k_deq = _fp8_forward(cu, N, P, layout, r, hq, hkv, d, bm, bn, q, k, v)
        ref = oracle.shard_forward(q_deq, k_deq, v.float().numpy(), cu, N, P, layout, r)
        o, lse = bufs["o"].float().cpu().numpy(), bufs["lse"].cpu().numpy()
        assert not np.isnan(o).any() and not np.isnan(lse).any(), r
        rep = {"o": max_abs(o, ref["o"]), "lse": max_abs(lse, ref["lse"])}
        _say("zero slices, shard", r, rep)
        assert rep["o"] <= O_ATOL and rep["lse"] <= LSE_ATOL, (r, rep)
