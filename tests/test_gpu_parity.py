"""GPU path (through the C ABI) against the fp64 oracle on the same seeded inputs.

Bars: tile lists bit-exact; O max-abs <= 2e-2; LSE max-abs <= 1e-3; the set of
-inf LSE rows of every partial identical; gradients max|g - ref| / max|ref|
<= 3e-2.  Small cases span several tiles, zero-length and one-token documents,
both shard layouts, GQA and both head dims; the benchmark's workloads are
compared on every row in test_gpu_workloads.py.
"""
import math
import sys

import numpy as np
import pytest
import torch

from _harness import Case, compare_backward, compare_forward, max_abs, rel_max
from paper_2606_30460_amd.shard_attention import to_sharded
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _rand_cu(rng, N, mean_len):
    lengths = []
    while sum(lengths) < N:
        lengths.append(int(rng.integers(1, 2 * mean_len)))
    lengths[-1] -= sum(lengths) - N
    cu = np.concatenate([[0], np.cumsum(lengths)])
    # a zero-length document and some one-token documents
    cu = np.sort(np.concatenate([cu, [cu[len(cu) // 2]], [1, 2, 3]]))
    return np.unique(cu) if rng.random() < 0.5 else cu


SMALL = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length
    (1024, 1, "contiguous", 4, 4, 64, 64, 64, 200),
    (2048, 2, "contiguous", 4, 2, 128, 128, 128, 300),
    (2048, 4, "zigzag", 8, 2, 128, 128, 64, 150),
    (4096, 4, "contiguous", 2, 1, 128, 64, 128, 900),
    (4096, 8, "zigzag", 4, 4, 64, 64, 64, 40),
    (2048, 2, "zigzag", 2, 2, 128, 64, 64, 5),
    (3072, 3, "contiguous", 6, 3, 64, 128, 64, 3000),
    (4096, 2, "zigzag", 4, 2, 128, 256, 128, 700),
    (4096, 4, "contiguous", 2, 2, 128, 256, 64, 300),
    # K/V heads a multiple of 8 with grouped query heads: the query heads of one K/V head are
    # placed on one XCD (groups of 2 and 8)
    (2048, 2, "zigzag", 16, 8, 128, 128, 128, 400),
    (2048, 2, "contiguous", 64, 8, 128, 128, 64, 250),
]


@pytest.mark.parametrize("case", SMALL)
def test_forward_small(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    rng = np.random.default_rng(N + P * 7 + hq)
    cu = _rand_cu(rng, N, mean)
    for r in sorted({0, P - 1, P // 2}):
        _say("forward small", case, "shard", r)
        c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=r)
        gpu = c.run_gpu()
        ref = c.run_oracle()
        compare_forward(gpu, ref)
        # executing chunk by chunk in ring order gives the identical bits
        gpu2 = c.run_gpu(ring_steps=True)
        assert np.array_equal(gpu2["o"], gpu["o"]) and np.array_equal(gpu2["lse"], gpu["lse"])


def test_forward_many_chunks():
    # 260 chunks: beyond what the direct-to-LDS kernel's packed tile descriptors hold, so 128-row
    # q-tiles of head_dim 128 run on the register-staged kernel; both shards' ends of the ring
    N, P = 260 * 128, 260
    cu = _rand_cu(np.random.default_rng(260), N, 1500)
    for r in (3, P - 1):
        _say("forward many chunks, shard", r)
        c = Case(cu, N, P, "contiguous", r, 2, 2, 128, 128, 128, seed=r)
        compare_forward(c.run_gpu(), c.run_oracle())


@pytest.mark.parametrize("split", [0, 1, 3])
def test_forward_split_runs(split):
    # long runs cut into pieces of at most `split` tiles (0: never) give the same result
    N, P = 4096, 2
    lengths = [3000, 40, 1, 1055]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    c = Case(cu, N, P, "contiguous", 1, 4, 2, 128, 128, 128, seed=9)
    gpu = c.run_gpu(max_run_tiles=split)
    ref = c.run_oracle()
    compare_forward(gpu, ref)
    sa = gpu["sa"]
    if split:
        assert sa.num_slots > P and len(sa.present) > len(sa.chunks_present)
    else:
        assert len(sa.present) == len(sa.chunks_present)


def test_forward_one_token_documents_exact():
    # a one-token document attends only to itself: O equals its V row bit for bit
    N, P = 1024, 2
    lengths = [1] * 300 + [200, 1, 1, 1, 300] + [1] * 221
    cu = np.concatenate([[0], np.cumsum(lengths)])
    assert cu[-1] == N
    c = Case(cu, N, P, "contiguous", 1, 4, 4, 128, 128, 128, seed=3)
    gpu = c.run_gpu()
    ref = c.run_oracle()
    compare_forward(gpu, ref)
    ones = [i for i in range(len(lengths)) if lengths[i] == 1]
    pos = [int(cu[i]) for i in ones if cu[i] >= N // 2]
    local = [p - N // 2 for p in pos]
    v = c.v.float().numpy()
    assert np.array_equal(gpu["o"][local], v[pos])
    q, k = c.q.float().numpy(), c.k.float().numpy()
    lse_exact = np.einsum("nhd,nhd->hn", q[pos], k[pos]) / math.sqrt(128)
    assert max_abs(gpu["lse"][:, local], lse_exact) <= 1e-5


def test_forward_zero_query_closed_form():
    # Q = 0: LSE_i = ln(i - start(i) + 1) and O_i is the mean of V over the document prefix
    N, P = 2048, 4
    lengths = [700, 1, 129, 64, 500, 654]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    c = Case(cu, N, P, "zigzag", 2, 4, 2, 128, 64, 64, seed=5, q_zero=True)
    gpu = c.run_gpu()
    import oracle
    pos = oracle.shard_positions(N, P, "zigzag", 2)
    start = oracle.doc_starts(cu)[pos]
    np.testing.assert_allclose(gpu["lse"], np.log(pos - start + 1.0)[None, :].repeat(4, 0), atol=1e-5, rtol=0)
    v = c.v.float().numpy().astype(np.float64)
    csum = np.concatenate([np.zeros((1, 2, 128)), np.cumsum(v, axis=0)])
    mean = (csum[pos + 1] - csum[start]) / (pos - start + 1.0)[:, None, None]
    assert max_abs(gpu["o"], np.repeat(mean, 2, axis=1)) <= 2e-2


@pytest.mark.parametrize("parts,d,n", [(1, 128, 300), (2, 128, 300), (2, 64, 17), (3, 128, 33), (4, 64, 300),
                                       (5, 128, 300), (9, 64, 45), (14, 128, 77), (64, 128, 40), (64, 64, 19)])
def test_merge_alone_matches_oracle_merge(parts, d, n):
    # the merge kernel fed the oracle's own partials: O within one bf16 rounding, LSE within 1e-5;
    # O rows of parts whose LSE is -inf hold NaN, so reading one would show
    from paper_2606_30460_amd import _lib as L
    import oracle
    rng = np.random.default_rng(11 + parts + n)
    hq = 3
    o_p = [rng.standard_normal((n, hq, d)) for _ in range(parts)]
    l_p = [rng.standard_normal((hq, n)) * 3 for _ in range(parts)]
    if parts > 1:
        l_p[1][:, ::3] = -np.inf
    if parts > 2:
        l_p[2][:, ::2] = -np.inf
    for p in range(parts):
        l_p[p][:, 7 % n] = -np.inf                  # a row with no part at all
    o_ref, l_ref = oracle.lse_merge(o_p, l_p)
    for p in range(parts):
        o_p[p][np.isneginf(l_p[p]).T] = np.nan      # never written by the forward: must not be read
    dev = torch.device("cuda")
    o_t = [torch.tensor(x, dtype=torch.float32, device=dev) for x in o_p]
    l_t = [torch.tensor(x, dtype=torch.float32, device=dev) for x in l_p]
    o_out = torch.empty(n, hq, d, dtype=torch.bfloat16, device=dev)
    l_out = torch.empty(hq, n, dtype=torch.float32, device=dev)
    L.lse_merge(o_t, l_t, n, hq, d, o_out, l_out)
    torch.cuda.synchronize()
    l_g = l_out.cpu().numpy()
    assert np.array_equal(np.isneginf(l_g), np.isneginf(l_ref))
    fin = np.isfinite(l_ref)
    assert max_abs(l_g[fin], l_ref[fin]) <= 1e-5
    o_g = o_out.float().cpu().numpy()
    ulp = np.abs(o_ref) * 2.0 ** -8 + 1e-30
    assert np.all(np.abs(o_g - o_ref) <= ulp + 1e-5)
    assert np.all(o_g[7 % n] == 0.0)


def test_doc_start_and_gather():
    from paper_2606_30460_amd import _lib as L
    from paper_2606_30460_amd.shard_attention import to_sharded
    import oracle
    cu = np.array([0, 0, 5, 5, 6, 100, 1000, 1024], dtype=np.int32)
    dev = torch.device("cuda")
    out = torch.empty(1024, dtype=torch.int32, device=dev)
    L.doc_start(torch.from_numpy(cu).to(dev), 1024, out)
    assert np.array_equal(out.cpu().numpy(), oracle.doc_starts(cu))
    for layout in ("contiguous", "zigzag"):
        x = torch.arange(1024 * 8, dtype=torch.float32, device=dev).view(1024, 8)
        sh = to_sharded(L.shard_desc(1024, 4, layout, 0, 1, 1), x).cpu().numpy()
        for r in range(4):
            assert np.array_equal(sh[r][:, 0] / 8, oracle.shard_positions(1024, 4, layout, r))


def test_forward_small_workload():
    # the 2048-token, six-document workload (SP degree 1) on every row; the larger workloads, with
    # the benchmark's executor path, are in test_gpu_workloads.py
    w = make_workload("c1")
    c = Case.from_workload(w)
    _say("workload c1 shard", c.shard)
    ref = c.run_oracle()
    rep = compare_forward(c.run_gpu(), ref)
    _say("c1 max errors", {k: round(v, 6) for k, v in rep.items() if k in ("o", "lse")})
    ex = c.run_executor()
    assert max_abs(ex["o"], ref["o"]) <= 2e-2 and max_abs(ex["lse"], ref["lse"]) <= 1e-3


# ---------------------------------------------------------------------------
# backward
# ---------------------------------------------------------------------------

SMALL_BWD = [
    # N, P, layout, hq, hkv, d, bm, bn, mean doc length
    (1024, 1, "contiguous", 2, 2, 64, 64, 64, 300),
    (2048, 2, "contiguous", 4, 2, 128, 128, 128, 300),
    (2048, 4, "zigzag", 4, 1, 128, 128, 64, 120),
    (4096, 4, "contiguous", 2, 2, 128, 64, 128, 5),
    # 256-row q-tiles (eight-wave dQ kernel, four 64-row sub-tiles per tile in dK/dV), GQA
    (4096, 2, "zigzag", 4, 2, 128, 256, 128, 700),
    (8192, 4, "contiguous", 8, 2, 128, 256, 64, 40),
    # K/V heads a multiple of 8 with grouped query heads (the dQ kernel's XCD placement)
    (2048, 2, "contiguous", 16, 8, 128, 128, 128, 300),
]


@pytest.mark.parametrize("case", SMALL_BWD)
def test_backward_small(case):
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    rng = np.random.default_rng(N + 3 * P + hq)
    cu = _rand_cu(rng, N, mean)
    for r in sorted({0, P - 1}):
        _say("backward small", case, "shard", r)
        c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=10 + r, backward=True)
        gpu = c.run_gpu()
        ref = c.run_oracle()
        compare_forward(gpu, ref["fwd"])
        rep = compare_backward(gpu, ref)
        _say(case, r, rep)


def test_backward_ring_steps_accumulate():
    """dQ accumulated over one call per ring step (each chunk's unsplit q-major runs), dK/dV per
    chunk, equals the one-pass result within rounding and meets the oracle."""
    from paper_2606_30460_amd import _lib as L
    N, P, layout, hq, hkv, d, bm, bn = 4096, 4, "contiguous", 4, 2, 128, 128, 128
    cu = np.array([0, 700, 2600, 2601, 4096], dtype=np.int32)
    r = 3
    c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=5, backward=True)
    gpu = c.run_gpu()
    ref = c.run_oracle()
    sa = gpu["sa"]
    dev = torch.device("cuda")
    q = to_sharded(sa.shard, c.q.to(dev))[r].contiguous()
    k, v = to_sharded(sa.shard, c.k.to(dev)), to_sharded(sa.shard, c.v.to(dev))
    d_o = to_sharded(sa.shard, c.do.to(dev))[r].contiguous()
    fwd = sa.alloc_forward()
    sa.forward(q, k, v, fwd)
    bwd = sa.alloc_backward()
    L.attn_bwd_preprocess(fwd["o"], d_o, sa.n, hq, d, bwd["delta"])
    tiles_q, runs_q, _ = L.plan_runs(sa.shard, sa.tiles, L.MAJOR_Q, 0)
    tq = torch.from_numpy(tiles_q.reshape(-1)).to(dev)
    for chunk in sa.chunks:
        sel = runs_q[runs_q[:, 0] == chunk]
        if len(sel):
            L.partial_attn_bwd_runs(sa.desc, q, k, v, d_o, fwd["lse"], bwd["delta"], sa.doc_start, None, None, tq,
                               torch.from_numpy(np.ascontiguousarray(sel).reshape(-1)).to(dev), bwd["dq_acc"],
                               bwd["dk_acc"], bwd["dv_acc"])
    torch.cuda.synchronize()
    dq = bwd["dq_acc"].cpu().numpy()
    rep = {"dq_vs_onepass": rel_max(dq, gpu["dq"]), "dq_vs_oracle": rel_max(dq, ref["dq"])}
    _say(rep)
    assert rep["dq_vs_onepass"] <= 1e-5 and rep["dq_vs_oracle"] <= 3e-2, rep



# ---------------------------------------------------------------------------
# the boundary's tile-list calls (hsap_partial_attn_fwd / _bwd on one chunk's tiles)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case", SMALL_BWD + [SMALL[2], SMALL[4]])
def test_tile_list_entry_points(case):
    """hsap_partial_attn_fwd / hsap_partial_attn_bwd called once per ring step with that chunk's
    tiles from hsap_plan (K/V of the chunk passed alone): each partial, the merge and the gradients
    against the oracle; the forward partials equal the run-based entry point's bit for bit (the
    same kernel over the same tiles per q-tile)."""
    from paper_2606_30460_amd import _lib as L
    from _harness import compare_tile_list
    N, P, layout, hq, hkv, d, bm, bn, mean = case
    rng = np.random.default_rng(N + 11 * P + hq)
    cu = _rand_cu(rng, N, mean)
    bwd = (d == 128 or bn == 64) and (bm <= 128 or d == 128)
    for r in sorted({0, P - 1}):
        _say("tile lists", case, "shard", r)
        c = Case(cu, N, P, layout, r, hq, hkv, d, bm, bn, seed=30 + r, backward=bwd)
        got = c.run_tile_list()
        ref = c.run_oracle()
        rep = compare_tile_list(got, ref["fwd"] if bwd else ref)
        runs = c.run_gpu(max_run_tiles=0)
        for step, ch in enumerate(got["chunks"]):
            if got["step_offsets"][step + 1] > got["step_offsets"][step]:
                fin = ~np.isneginf(runs["lse_part"][ch])
                assert np.array_equal(got["lse_part"][ch], runs["lse_part"][ch])
                assert np.array_equal(got["o_part"][ch][fin.T], runs["o_part"][ch][fin.T])
        if bwd:
            rep.update(compare_backward(got, ref))
        _say({k: round(v, 6) for k, v in rep.items() if not k.startswith(("o_part", "lse_part"))})
