"""Pins for the fp64 oracle: brute force, closed forms, library routines, invariants.

Each test states which property of the paper's method (or of the mathematics)
fixes the expected value, so that a wrong mask bound, a dropped term, a wrong
sign or a transposed operand inside the oracle fails at least one of them.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle.plan import KIND_FULL, KIND_MASKED, plan_shard, tile_pair_counts, tile_pair_counts_bruteforce

ATOL = 1e-12


def _rand_cu(rng, total):
    """Random cumulative lengths over ``total`` tokens.

    Cut points are drawn with replacement, so repeated cuts give zero-length
    documents and neighbouring cuts give one-token documents.
    """
    ncut = int(rng.integers(0, max(1, total // 3) + 1))
    cuts = rng.integers(0, total + 1, size=ncut)
    return np.sort(np.concatenate([[0, total], cuts])).astype(np.int64)


def _rand(rng, *shape):
    return rng.standard_normal(shape)


# ---------------------------------------------------------------------------
# P1: brute-force dense masked softmax (pair-by-pair mask, scipy softmax)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
def test_p1_bruteforce_dense(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 48))
    cu = _rand_cu(rng, N)
    hkv = int(rng.choice([1, 2]))
    hq = hkv * int(rng.choice([1, 2, 3]))
    d = int(rng.choice([3, 8]))
    q, k, v = _rand(rng, N, hq, d), _rand(rng, N, hkv, d), _rand(rng, N, hkv, d)
    # arbitrary query subset and key subset, in arbitrary order
    q_pos = rng.permutation(N)[: int(rng.integers(1, N + 1))]
    k_pos = rng.permutation(N)[: int(rng.integers(1, N + 1))]
    scale = 1.0 / math.sqrt(d)
    o, lse = oracle.attention_fwd(q[q_pos], k[k_pos], v[k_pos], q_pos, k_pos, cu)
    mask = oracle.allowed_mask_dense(cu, q_pos, k_pos)
    grp = hq // hkv
    for a in range(len(q_pos)):
        for h in range(hq):
            g = h // grp
            sel = np.nonzero(mask[a])[0]
            if sel.size == 0:
                assert lse[h, a] == -np.inf
                assert np.all(o[a, h] == 0.0)
                continue
            s = np.array([q[q_pos[a], h] @ k[k_pos[b], g] for b in sel]) * scale
            w = scipy.special.softmax(s)
            np.testing.assert_allclose(lse[h, a], scipy.special.logsumexp(s), atol=ATOL, rtol=0)
            np.testing.assert_allclose(o[a, h], w @ v[k_pos[sel], g], atol=ATOL, rtol=0)


# ---------------------------------------------------------------------------
# P2: packing causes no cross-contamination: equals each document run alone
#     through torch's causal SDPA (float64, CPU)
# ---------------------------------------------------------------------------

def _sdpa_causal(q, k, v):
    """torch SDPA on one document; q [L, H, d] -> [L, H, d]."""
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2)[None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    return out[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("seed", range(4))
def test_p2_no_cross_contamination(seed):
    rng = np.random.default_rng(100 + seed)
    lengths = [int(x) for x in rng.integers(1, 40, size=6)]
    N, H, d = sum(lengths), 3, 16
    cu = np.concatenate([[0], np.cumsum(lengths)])
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o, _ = oracle.attention_fwd(q, k, v, pos, pos, cu)
    ref = np.concatenate([_sdpa_causal(q[a:b], k[a:b], v[a:b]) for a, b in zip(cu[:-1], cu[1:])])
    np.testing.assert_allclose(o, ref, atol=1e-12, rtol=0)
    # permuting the documents permutes the outputs
    perm = rng.permutation(len(lengths))
    segs = [(cu[i], cu[i + 1]) for i in perm]
    idx = np.concatenate([np.arange(a, b) for a, b in segs])
    cu2 = np.concatenate([[0], np.cumsum([lengths[i] for i in perm])])
    o2, _ = oracle.attention_fwd(q[idx], k[idx], v[idx], pos, pos, cu2)
    np.testing.assert_allclose(o2, o[idx], atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# P3: a one-token document attends only to itself
# ---------------------------------------------------------------------------

def test_p3_one_token_document():
    rng = np.random.default_rng(7)
    lengths = [5, 1, 9, 1, 1, 4]
    N, H, d = sum(lengths), 2, 8
    cu = np.concatenate([[0], np.cumsum(lengths)])
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o, lse = oracle.attention_fwd(q, k, v, pos, pos, cu)
    for i in (5, 15, 16):                         # the one-token documents
        for h in range(H):
            assert np.array_equal(o[i, h], v[i, h])
            # the only score of the row is its own, so LSE is that score (up to rounding order)
            np.testing.assert_allclose(lse[h, i], (q[i, h] @ k[i, h]) / math.sqrt(d), rtol=1e-15, atol=1e-15)


# ---------------------------------------------------------------------------
# P4: closed form with Q == 0: uniform weights over [start(i), i]
# ---------------------------------------------------------------------------

def test_p4_zero_query_closed_form():
    rng = np.random.default_rng(8)
    lengths = [3, 1, 17, 8, 1, 30]
    N, H, d = sum(lengths), 2, 4
    cu = np.concatenate([[0], np.cumsum(lengths)])
    q = np.zeros((N, H, d))
    k, v = _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o, lse = oracle.attention_fwd(q, k, v, pos, pos, cu)
    csum = np.concatenate([np.zeros((1, H, d)), np.cumsum(v, axis=0)])
    for a, b in zip(cu[:-1], cu[1:]):
        for i in range(a, b):
            count = i - a + 1
            np.testing.assert_allclose(lse[:, i], math.log(count), atol=ATOL, rtol=0)
            np.testing.assert_allclose(o[i], (csum[i + 1] - csum[a]) / count, atol=ATOL, rtol=0)


# ---------------------------------------------------------------------------
# P5: merging partials over ANY chunking equals the unchunked result
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(5))
def test_p5_merge_chunking_invariance(seed):
    rng = np.random.default_rng(200 + seed)
    N = int(rng.integers(8, 64))
    cu = _rand_cu(rng, N)
    H, d = 2, 8
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o_ref, lse_ref = oracle.attention_fwd(q, k, v, pos, pos, cu)
    # random chunking of the key positions: includes singletons and chunks that split documents
    nparts = int(rng.integers(1, min(N, 9) + 1))
    label = rng.integers(0, nparts, size=N)
    label[: nparts] = np.arange(nparts)            # every part non-empty
    parts = [np.nonzero(label == p)[0] for p in range(nparts)]
    if seed == 0:
        parts = [np.array([j]) for j in range(N)]  # chunk size 1
    o_p, l_p = [], []
    for kp in parts:
        o_c, l_c = oracle.attention_fwd(q, k[kp], v[kp], pos, kp, cu)
        o_p.append(o_c)
        l_p.append(l_c)
    # add a partial whose rows are all -inf (a chunk that shares no document)
    o_p.append(np.full_like(o_ref, 123.0))
    l_p.append(np.full_like(lse_ref, -np.inf))
    order = rng.permutation(len(o_p))
    o_m, l_m = oracle.lse_merge([o_p[i] for i in order], [l_p[i] for i in order])
    np.testing.assert_allclose(o_m, o_ref, atol=ATOL, rtol=0)
    np.testing.assert_allclose(l_m, lse_ref, atol=ATOL, rtol=0)
    # associativity: merge of merges
    half = len(o_p) // 2
    a = oracle.lse_merge(o_p[:half] or [o_p[0]], l_p[:half] or [l_p[0]]) if half else None
    if a is not None:
        b = oracle.lse_merge(o_p[half:], l_p[half:])
        o_ab, l_ab = oracle.lse_merge([a[0], b[0]], [a[1], b[1]])
        np.testing.assert_allclose(o_ab, o_ref, atol=ATOL, rtol=0)
        np.testing.assert_allclose(l_ab, lse_ref, atol=ATOL, rtol=0)


def test_p5_merge_all_neg_inf_rows():
    o = [np.ones((3, 1, 2)), np.full((3, 1, 2), 7.0)]
    l = [np.full((1, 3), -np.inf), np.full((1, 3), -np.inf)]
    o_m, l_m = oracle.lse_merge(o, l)
    assert np.all(o_m == 0.0) and np.all(l_m == -np.inf)


# ---------------------------------------------------------------------------
# P6: reductions to textbook causal attention
# ---------------------------------------------------------------------------

def test_p6_single_document_is_causal_sdpa():
    rng = np.random.default_rng(9)
    N, H, d = 70, 3, 16
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o, _ = oracle.attention_fwd(q, k, v, pos, pos, [0, N])
    np.testing.assert_allclose(o, _sdpa_causal(q, k, v), atol=1e-12, rtol=0)


def test_p6_uniform_documents_are_batched_causal_sdpa():
    rng = np.random.default_rng(10)
    L, B, H, d = 12, 5, 2, 8
    N = L * B
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    o, _ = oracle.attention_fwd(q, k, v, pos, pos, np.arange(0, N + 1, L))
    tq = torch.from_numpy(q.reshape(B, L, H, d)).permute(0, 2, 1, 3)
    tk = torch.from_numpy(k.reshape(B, L, H, d)).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v.reshape(B, L, H, d)).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    np.testing.assert_allclose(o, ref.permute(0, 2, 1, 3).reshape(N, H, d).numpy(), atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# P7: GQA equals MHA with K/V heads repeated; gradients group-summed
# ---------------------------------------------------------------------------

def test_p7_gqa_equals_repeated_mha():
    rng = np.random.default_rng(11)
    N, hkv, grp, d = 40, 2, 3, 8
    hq = hkv * grp
    cu = np.array([0, 7, 8, 25, 40])
    q, k, v, do = _rand(rng, N, hq, d), _rand(rng, N, hkv, d), _rand(rng, N, hkv, d), _rand(rng, N, hq, d)
    k_rep, v_rep = np.repeat(k, grp, axis=1), np.repeat(v, grp, axis=1)
    pos = np.arange(N)
    o_g, l_g = oracle.attention_fwd(q, k, v, pos, pos, cu)
    o_m, l_m = oracle.attention_fwd(q, k_rep, v_rep, pos, pos, cu)
    np.testing.assert_allclose(o_g, o_m, atol=ATOL, rtol=0)
    np.testing.assert_allclose(l_g, l_m, atol=ATOL, rtol=0)
    delta = np.einsum("nhd,nhd->hn", do, o_g)
    dq_g, dk_g, dv_g = oracle.attention_bwd(q, k, v, do, l_g, delta, pos, pos, cu)
    dq_m, dk_m, dv_m = oracle.attention_bwd(q, k_rep, v_rep, do, l_m, delta, pos, pos, cu)
    np.testing.assert_allclose(dq_g, dq_m, atol=ATOL, rtol=0)
    np.testing.assert_allclose(dk_g, dk_m.reshape(N, hkv, grp, d).sum(2), atol=ATOL, rtol=0)
    np.testing.assert_allclose(dv_g, dv_m.reshape(N, hkv, grp, d).sum(2), atol=ATOL, rtol=0)


# ---------------------------------------------------------------------------
# P8: backward = derivative of the forward (finite differences, torch autograd)
# ---------------------------------------------------------------------------

def _loss_and_grads(q, k, v, w, cu, pos):
    o, lse = oracle.attention_fwd(q, k, v, pos, pos, cu)
    delta = np.einsum("nhd,nhd->hn", w, o)
    grads = oracle.attention_bwd(q, k, v, w, lse, delta, pos, pos, cu)
    return float(np.sum(o * w)), grads


def test_p8_finite_differences():
    rng = np.random.default_rng(12)
    N, hkv, grp, d = 14, 1, 2, 4
    hq = hkv * grp
    cu = np.array([0, 1, 6, 6, 14])
    q, k, v, w = _rand(rng, N, hq, d), _rand(rng, N, hkv, d), _rand(rng, N, hkv, d), _rand(rng, N, hq, d)
    pos = np.arange(N)
    _, (dq, dk, dv) = _loss_and_grads(q, k, v, w, cu, pos)
    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        fd = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}
            args_m = {"q": q, "k": k, "v": v}
            args_p[name], args_m[name] = xp, xm
            lp = np.sum(oracle.attention_fwd(args_p["q"], args_p["k"], args_p["v"], pos, pos, cu)[0] * w)
            lm = np.sum(oracle.attention_fwd(args_m["q"], args_m["k"], args_m["v"], pos, pos, cu)[0] * w)
            fd[idx] = (lp - lm) / (2 * h)
        rel = np.max(np.abs(fd - g)) / np.max(np.abs(g))
        assert rel < 1e-7, (name, rel)


def test_p8_torch_autograd():
    rng = np.random.default_rng(13)
    N, H, d = 30, 2, 8
    cu = np.array([0, 4, 5, 19, 30])
    q, k, v, w = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    _, (dq, dk, dv) = _loss_and_grads(q, k, v, w, cu, pos)
    doc = np.repeat(np.arange(len(cu) - 1), np.diff(cu))
    allowed = torch.from_numpy((doc[:, None] == doc[None, :]) & (pos[None, :] <= pos[:, None]))
    tq, tk, tv = (torch.from_numpy(x.copy()).requires_grad_() for x in (q, k, v))
    s = torch.einsum("ihd,jhd->hij", tq, tk) / math.sqrt(d)
    p = torch.softmax(s.masked_fill(~allowed, float("-inf")), dim=-1)
    o = torch.einsum("hij,jhd->ihd", p, tv)
    (o * torch.from_numpy(w)).sum().backward()
    for ours, ref in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        np.testing.assert_allclose(ours, ref.numpy(), atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# P9: backward invariants
# ---------------------------------------------------------------------------

def test_p9_backward_invariants():
    rng = np.random.default_rng(14)
    N, H, d = 50, 2, 8
    cu = np.array([0, 1, 13, 13, 37, 50])
    q, k, v, w = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    pos = np.arange(N)
    _, (dq, dk, dv) = _loss_and_grads(q, k, v, w, cu, pos)
    for a, b in zip(cu[:-1], cu[1:]):
        if a == b:
            continue
        np.testing.assert_allclose(dk[a:b].sum(0), 0.0, atol=1e-12)
        np.testing.assert_allclose(dv[a:b].sum(0), w[a:b].sum(0), atol=1e-12)
    # a constant added to every key shifts each row's scores uniformly
    c = rng.standard_normal((1, H, d))
    o1, l1 = oracle.attention_fwd(q, k, v, pos, pos, cu)
    o2, l2 = oracle.attention_fwd(q, k + c, v, pos, pos, cu)
    np.testing.assert_allclose(o2, o1, atol=1e-12)
    np.testing.assert_allclose(l2 - l1, np.einsum("nhd,hd->hn", q, c[0]) / math.sqrt(d), atol=1e-12)
    _, (dq2, _, _) = _loss_and_grads(q, k + c, v, w, cu, pos)
    np.testing.assert_allclose(dq2, dq, atol=1e-12)


# ---------------------------------------------------------------------------
# Shard bookkeeping: shard outputs assemble to the unsharded result
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
def test_shards_assemble_unsharded(layout):
    rng = np.random.default_rng(15)
    P, N, hq, hkv, d = 4, 64, 4, 2, 8
    cu = _rand_cu(rng, N)
    q, k, v, do = _rand(rng, N, hq, d), _rand(rng, N, hkv, d), _rand(rng, N, hkv, d), _rand(rng, N, hq, d)
    pos = np.arange(N)
    o_ref, l_ref = oracle.attention_fwd(q, k, v, pos, pos, cu)
    delta = np.einsum("nhd,nhd->hn", do, o_ref)
    dq_ref, dk_ref, dv_ref = oracle.attention_bwd(q, k, v, do, l_ref, delta, pos, pos, cu)
    seen = np.zeros(N, dtype=int)
    dk_sum = np.zeros_like(dk_ref)
    dv_sum = np.zeros_like(dv_ref)
    for r in range(P):
        qp = oracle.shard_positions(N, P, layout, r)
        seen[qp] += 1
        fwd = oracle.shard_forward(q, k, v, cu, N, P, layout, r)
        assert fwd["chunks"] == [(r - s) % P for s in range(P)]
        np.testing.assert_allclose(fwd["o"], o_ref[qp], atol=ATOL, rtol=0)
        np.testing.assert_allclose(fwd["lse"], l_ref[:, qp], atol=ATOL, rtol=0)
        bwd = oracle.shard_backward(q, k, v, do, cu, N, P, layout, r)
        np.testing.assert_allclose(bwd["dq"], dq_ref[qp], atol=1e-12, rtol=0)
        for c in range(P):
            kp = oracle.shard_positions(N, P, layout, c)
            dk_sum[kp] += bwd["dk"][c]
            dv_sum[kp] += bwd["dv"][c]
    assert np.all(seen == 1)
    np.testing.assert_allclose(dk_sum, dk_ref, atol=1e-12, rtol=0)
    np.testing.assert_allclose(dv_sum, dv_ref, atol=1e-12, rtol=0)


def test_zigzag_layout_pieces_and_balance():
    P, N = 4, 64
    m = N // (2 * P)
    for r in range(P):
        pos = oracle.shard_positions(N, P, "zigzag", r)
        assert list(pos[:m]) == list(range(r * m, (r + 1) * m))
        assert list(pos[m:]) == list(range((2 * P - 1 - r) * m, (2 * P - r) * m))
    # one causal document over the whole sequence: zigzag balances the pairs exactly
    pairs = oracle.useful_pairs_all_shards([0, N], N, P, "zigzag")
    assert len(set(pairs.tolist())) == 1
    assert int(pairs.sum()) == N * (N + 1) // 2
    contiguous = oracle.useful_pairs_all_shards([0, N], N, P, "contiguous")
    assert list(contiguous) == sorted(contiguous) and contiguous[0] < contiguous[-1]


# ---------------------------------------------------------------------------
# P10 / P11: planner counts, classification and the pair-count identity
# ---------------------------------------------------------------------------

CASES = [
    # (N, P, layout, BM, BN, cu)
    (64, 1, "contiguous", 16, 16, [0, 64]),
    (64, 2, "contiguous", 16, 32, [0, 1, 2, 17, 17, 40, 64]),
    (128, 4, "zigzag", 16, 16, [0, 16, 32, 33, 90, 128]),
    (128, 8, "contiguous", 16, 16, list(range(0, 129, 16))),   # a document equal to a tile
    (128, 2, "zigzag", 32, 16, [0, 128]),                      # a document crossing every chunk
]


@pytest.mark.parametrize("case", CASES)
def test_p10_counts_bruteforce_vs_rowwise(case):
    N, P, layout, bm, bn, cu = case
    for r in range(P):
        for c in range(P):
            a = tile_pair_counts_bruteforce(cu, N, P, layout, r, c, bm, bn)
            b = tile_pair_counts(cu, N, P, layout, r, c, bm, bn)
            assert np.array_equal(a, b)


@pytest.mark.parametrize("seed", range(6))
def test_p10_random_counts(seed):
    rng = np.random.default_rng(300 + seed)
    P = int(rng.choice([1, 2, 4]))
    layout = str(rng.choice(["contiguous", "zigzag"]))
    bm, bn = int(rng.choice([8, 16])), int(rng.choice([8, 16]))
    N = 2 * P * 32
    cu = _rand_cu(rng, N)
    r = int(rng.integers(0, P))
    for c in range(P):
        assert np.array_equal(tile_pair_counts_bruteforce(cu, N, P, layout, r, c, bm, bn),
                              tile_pair_counts(cu, N, P, layout, r, c, bm, bn))


@pytest.mark.parametrize("case", CASES)
def test_p11_pair_identity_and_kinds(case):
    N, P, layout, bm, bn, cu = case
    lengths = np.diff(cu)
    expect = int(np.sum(lengths * (lengths + 1) // 2))
    total = 0
    per_shard = oracle.useful_pairs_all_shards(cu, N, P, layout)
    for r in range(P):
        plan = plan_shard(cu, N, P, layout, r, bm, bn)
        total += int(plan["useful_pairs"].sum())
        assert int(plan["useful_pairs"].sum()) == int(per_shard[r])
        kinds = plan["tiles"][:, 3]
        assert np.all((kinds == KIND_FULL) == (plan["pairs"] == bm * bn))
        assert np.all((kinds == KIND_FULL) | (kinds == KIND_MASKED))
        assert np.all(plan["pairs"] > 0)
        # canonical order: ring step, then q-tile, then k-tile
        offs = plan["step_offsets"]
        for s in range(P):
            seg = plan["tiles"][offs[s]:offs[s + 1]]
            assert np.all(seg[:, 0] == (r - s) % P)
            keys = seg[:, 1].astype(np.int64) * 100000 + seg[:, 2]
            assert np.all(np.diff(keys) > 0)
    assert total == expect


@pytest.mark.parametrize("tile", [2, 16])
def test_p11_causal_single_doc_tile_kinds(tile):
    # one document, one shard: tiles on the diagonal are MASKED, below it FULL, above EMPTY.
    # With 2x2 tiles a diagonal tile holds 3 of its 4 pairs: one short of FULL.
    plan = plan_shard([0, 64], 64, 1, "contiguous", 0, tile, tile)
    got = {(int(t[1]), int(t[2])): int(t[3]) for t in plan["tiles"]}
    nt = 64 // tile
    for t in range(nt):
        for u in range(nt):
            if u > t:
                assert (t, u) not in got
            elif u == t:
                assert got[(t, u)] == KIND_MASKED
            else:
                assert got[(t, u)] == KIND_FULL
    assert int(plan["useful_pairs"][0]) == 64 * 65 // 2


# ---------------------------------------------------------------------------
# P12: rows with LSE = -inf in a partial are exactly the rows with no allowed key
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
def test_p12_neg_inf_structure(layout):
    rng = np.random.default_rng(16)
    P, N, H, d = 4, 64, 2, 4
    cu = _rand_cu(rng, N)
    q, k, v = _rand(rng, N, H, d), _rand(rng, N, H, d), _rand(rng, N, H, d)
    for r in range(P):
        fwd = oracle.shard_forward(q, k, v, cu, N, P, layout, r)
        qp = fwd["q_pos"]
        for c, lse_c in zip(fwd["chunks"], fwd["lse_parts"]):
            kp = oracle.shard_positions(N, P, layout, c)
            none = ~oracle.allowed_mask_dense(cu, qp, kp).any(axis=1)
            for h in range(H):
                assert np.array_equal(np.isneginf(lse_c[h]), none)
        assert np.all(np.isfinite(fwd["lse"]))        # the diagonal is always allowed


# ---------------------------------------------------------------------------
# Block loads of every shard and the Q-transfer rebalance
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("seed", range(3))
def test_load_matrix_counts_dense_mask(layout, seed):
    # every block's pair count is the number of allowed (query, key) pairs of the dense mask;
    # each shard's row sums to the closed form sum_i (i - start(i) + 1); tiles exist iff pairs do
    rng = np.random.default_rng(300 + seed)
    P, bm, bn = 4, 8, 4
    N = 2 * P * 16
    cu = _rand_cu(rng, N)
    tiles, pairs = oracle.load_matrix(cu, N, P, layout, bm, bn)
    for r in range(P):
        qp = oracle.shard_positions(N, P, layout, r)
        for c in range(P):
            kp = oracle.shard_positions(N, P, layout, c)
            assert pairs[r, c] == int(oracle.allowed_mask_dense(cu, qp, kp).sum())
            assert (tiles[r, c] > 0) == (pairs[r, c] > 0)
            assert pairs[r, c] <= tiles[r, c] * bm * bn
    assert np.array_equal(pairs.sum(axis=1), oracle.useful_pairs_all_shards(cu, N, P, layout))


def _check_assignment(cost, exec_rank, load):
    P = cost.shape[0]
    expect = np.zeros(P, dtype=np.int64)
    for r in range(P):
        assert exec_rank[r, r] == r
        for c in range(P):
            assert exec_rank[r, c] in (r, c)
            if cost[r, c] == 0:
                assert exec_rank[r, c] == r
            expect[exec_rank[r, c]] += cost[r, c]
    assert np.array_equal(load, expect)
    assert int(load.sum()) == int(cost.sum())


def _best_max_load(cost):
    """Smallest achievable maximum load, by trying every assignment of the movable blocks."""
    P = cost.shape[0]
    movable = [(r, c) for r in range(P) for c in range(P) if r != c and cost[r, c] > 0]
    best = None
    for bits in range(1 << len(movable)):
        load = np.diag(cost).astype(np.int64).copy()
        for i, (r, c) in enumerate(movable):
            load[c if bits >> i & 1 else r] += cost[r, c]
        best = int(load.max()) if best is None else min(best, int(load.max()))
    return best, len(movable)


def test_q_transfer_balance_worked_example():
    # Lower-triangular costs (causal, contiguous).  Ring loads [4, 9, 14].  Rank 2 gives: (2, 0)
    # w 5 to rank 0 leaves max(9, 9) = 9, (2, 1) w 7 to rank 1 would leave max(7, 16): take (2, 0)
    # -> [9, 9, 9].  Rank 0 (lowest of the equals) holds (2, 0) w 5; back to rank 2: 9 + 5 is
    # not below 9, so it stops.
    cost = np.array([[4, 0, 0], [6, 3, 0], [5, 7, 2]])
    exec_rank, load = oracle.q_transfer_balance(cost)
    assert load.tolist() == [9, 9, 9]
    assert exec_rank.tolist() == [[0, 0, 0], [1, 1, 1], [0, 2, 2]]   # empty blocks keep their row
    _check_assignment(cost, exec_rank, load)
    assert _best_max_load(cost)[0] == 9


def test_q_transfer_balance_one_causal_document():
    # one document over four contiguous shards of 8 x 8 tiles: diagonal blocks 36, below 64.
    # Ring loads [36, 100, 164, 228]; rank 3 gives (3, 0) to rank 0 (max(164, 100) = 164, the
    # same as (3, 1) -> rank 1 but lower c): [100, 100, 164, 164]; rank 2 then has no move
    # (100 + 64 is not below 164).  Six equal blocks on four ranks: 164 is the optimum.
    cost = np.array([[36, 0, 0, 0], [64, 36, 0, 0], [64, 64, 36, 0], [64, 64, 64, 36]])
    exec_rank, load = oracle.q_transfer_balance(cost)
    assert load.tolist() == [100, 100, 164, 164]
    assert exec_rank[3].tolist() == [0, 3, 3, 3] and exec_rank[2].tolist() == [2, 2, 2, 2]
    _check_assignment(cost, exec_rank, load)
    assert _best_max_load(cost)[0] == 164


@pytest.mark.parametrize("seed", range(40))
def test_q_transfer_balance_against_every_assignment(seed):
    rng = np.random.default_rng(900 + seed)
    P = int(rng.integers(1, 5))
    cost = rng.integers(0, 20, size=(P, P)) * (rng.random((P, P)) < 0.6)
    exec_rank, load = oracle.q_transfer_balance(cost)
    _check_assignment(cost, exec_rank, load)
    best, movable = _best_max_load(cost)
    assert best <= int(load.max()) <= int(cost.sum(axis=1).max())   # never worse than the ring
    if movable <= 1:   # one decision: the search finds the better side
        assert int(load.max()) == best


# ---------------------------------------------------------------------------
# Batches of packed sequences
# ---------------------------------------------------------------------------

def test_batch_of_one_is_the_single_sequence():
    rng = np.random.default_rng(77)
    P, N, H, d = 4, 64, 2, 4
    cu = _rand_cu(rng, N)
    q, k, v, do = (_rand(rng, N, H, d) for _ in range(4))
    for layout in ("contiguous", "zigzag"):
        for r in range(P):
            one = oracle.shard_forward(q, k, v, cu, N, P, layout, r)
            bat = oracle.batch_shard_forward(q, k, v, cu, N, 1, P, layout, r)
            assert np.array_equal(bat["o"], one["o"]) and np.array_equal(bat["lse"], one["lse"])
            p1, pb = plan_shard(cu, N, P, layout, r, 8, 4), oracle.batch_plan_shard(cu, N, 1, P, layout, r, 8, 4)
            assert np.array_equal(p1["tiles"], pb["tiles"]) and np.array_equal(p1["step_offsets"], pb["step_offsets"])
        g1 = oracle.shard_backward(q, k, v, do, cu, N, P, layout, 1)
        gb = oracle.batch_shard_backward(q, k, v, do, cu, N, 1, P, layout, 1)
        assert all(np.array_equal(g1[x], gb[x]) for x in ("dq", "dk", "dv"))


def test_batch_of_copies_gives_copies():
    rng = np.random.default_rng(78)
    P, N, H, d = 2, 32, 2, 4
    cu = _rand_cu(rng, N)
    q, k, v = (_rand(rng, N, H, d) for _ in range(3))
    cu2 = np.concatenate([cu, cu[1:] + N])
    q2, k2, v2 = (np.concatenate([x, x]) for x in (q, k, v))
    n = N // P
    for layout in ("contiguous", "zigzag"):
        for r in range(P):
            res = oracle.batch_shard_forward(q2, k2, v2, cu2, N, 2, P, layout, r)
            assert np.array_equal(res["o"][:n], res["o"][n:]) and np.array_equal(res["lse"][:, :n], res["lse"][:, n:])


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
def test_batch_tiles_bruteforce(layout):
    # the batch's tiles classify the concatenated sequence's allowed pairs over the batched row maps
    rng = np.random.default_rng(79)
    P, N, B, bm, bn = 2, 64, 3, 8, 4
    cus = [_rand_cu(rng, N) for _ in range(B)]
    cu = np.concatenate([cus[0]] + [c[1:] + b * N for b, c in enumerate(cus) if b > 0])
    n = N // P

    def rows(x):      # global positions of local rows b*n + l of shard x
        return np.concatenate([oracle.shard_positions(N, P, layout, x) + b * N for b in range(B)])

    for r in range(P):
        plan = oracle.batch_plan_shard(cu, N, B, P, layout, r, bm, bn)
        got = {(int(t[0]), int(t[1]), int(t[2])): int(t[3]) for t in plan["tiles"]}
        expect = {}
        qp = rows(r)
        for c in range(P):
            kp = rows(c)
            mask = oracle.allowed_mask_dense(cu, qp, kp)
            for t in range(B * n // bm):
                for u in range(B * n // bn):
                    cnt = int(mask[t * bm:(t + 1) * bm, u * bn:(u + 1) * bn].sum())
                    if cnt:
                        expect[(c, t, u)] = KIND_FULL if cnt == bm * bn else KIND_MASKED
        assert got == expect


# ---------------------------------------------------------------------------
# fp8 (e4m3) quantisation of Q and K
# ---------------------------------------------------------------------------

def test_fp8_worked_example():
    # amax 3 -> inv = 448 / 3 = 149.33: 1 -> 149.33 -> nearest e4m3 144 = 2^7 * 1.125 -> 0 1110 001;
    # -0.5 -> -74.67 -> -72 = -(2^6 * 1.125) -> 1 1101 001; 0.25 -> 37.33 -> 36 = 2^5 * 1.125 -> 0 1100 001;
    # 3 -> 448 = 2^8 * 1.75 -> 0 1111 110
    x = np.array([1.0, -0.5, 0.25, 3.0], dtype=np.float32).reshape(1, 4, 1, 1)
    codes, scale = oracle.quantize_fp8(x)
    assert codes.ravel().tolist() == [0x71, 0xE9, 0x61, 0x7E]
    assert scale[0, 0] == np.float32(3.0) / np.float32(448.0)


def test_fp8_decode_every_code():
    # e4m3 (bias 7, 3 mantissa bits): normal 2^(e-7) (1 + m/8), subnormal 2^-6 m/8; 0x7F / 0xFF are NaN
    codes = np.arange(256, dtype=np.uint8)
    got = oracle.decode_fp8(codes)
    for c in range(256):
        s, e, m = c >> 7, (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            assert np.isnan(got[c])
            continue
        mag = 2.0 ** (e - 7) * (1 + m / 8) if e else 2.0 ** -6 * (m / 8)
        assert got[c] == (-mag if s else mag)


def test_fp8_round_trip_and_amax():
    rng = np.random.default_rng(81)
    x = (rng.standard_normal((3, 40, 2, 16)) * np.array([1e-3, 5.0])[None, None, :, None]).astype(np.float32)
    x[1, :, 0, :] = 0.0                                   # a group with amax 0
    codes, scale = oracle.quantize_fp8(x)
    deq = oracle.dequantize_fp8(codes, scale)
    assert np.all(codes[1, :, 0, :] == 0) and scale[1, 0] == 0
    for g in range(3):
        for h in range(2):
            a = np.abs(x[g, :, h, :])
            if a.max() == 0:
                continue
            i = np.unravel_index(np.argmax(a), a.shape)
            assert codes[g, i[0], h, i[1]] & 0x7F == 0x7E          # the amax element lands on +-448
            # round trip: within half an e4m3 step (2^-4 relative for normals, 2^-10 absolute below)
            y = np.abs(x[g, :, h, :]) / scale[g, h]
            step = np.where(y >= 2.0 ** -6, 2.0 ** (np.floor(np.log2(np.maximum(y, 2.0 ** -6))) - 3), 2.0 ** -9)
            assert np.all(np.abs(deq[g, :, h, :] - x[g, :, h, :]) <= 0.5 * step * scale[g, h] * (1 + 1e-6))
