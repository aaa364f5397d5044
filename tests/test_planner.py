"""The C++ host planner (through the C ABI) against the oracle's tile classification, bit for bit.

The oracle classifies tiles by counting allowed pairs row by row (itself pinned
to brute-force pair classification); the library plans by interval
arithmetic.  Lists, ring-step offsets and per-step pair counts must be equal.
"""
import numpy as np
import pytest

import oracle
from oracle.plan import plan_shard, tile_pair_counts_bruteforce
from paper_2606_30460_amd import _lib as L
from workloads import make_workload


def _compare(cu, N, P, layout, r, bm, bn, counter=None):
    ref = plan_shard(cu, N, P, layout, r, bm, bn, **({"counter": counter} if counter else {}))
    got = L.plan(cu, L.shard_desc(N, P, layout, r, bm, bn))
    assert np.array_equal(got["tiles"], ref["tiles"])
    assert np.array_equal(got["step_offsets"], ref["step_offsets"])
    assert np.array_equal(got["useful_pairs"], ref["useful_pairs"])
    return got


def _rand_cu(rng, N):
    ncut = int(rng.integers(0, max(2, N // 8)))
    cuts = rng.integers(0, N + 1, size=ncut)
    return np.sort(np.concatenate([[0, N], cuts])).astype(np.int32)


@pytest.mark.parametrize("seed", range(40))
def test_random_against_bruteforce(seed):
    rng = np.random.default_rng(1000 + seed)
    P = int(rng.choice([1, 2, 4, 8, 16]))
    layout = str(rng.choice(["contiguous", "zigzag"]))
    bm, bn = int(rng.choice([16, 32, 64, 128])), int(rng.choice([16, 32, 64, 128]))
    split = 2 * P if layout == "zigzag" else P
    N = split * max(bm, bn) * int(rng.integers(1, 3))
    if N > 4096:
        N = split * max(bm, bn)
    cu = _rand_cu(rng, N)
    r = int(rng.integers(0, P))
    _compare(cu, N, P, layout, r, bm, bn, counter=tile_pair_counts_bruteforce if N <= 1024 else None)


EDGE = [
    # one-token documents everywhere
    (256, 4, "contiguous", 16, 16, np.arange(0, 257)),
    # zero-length documents
    (256, 2, "zigzag", 32, 32, [0, 0, 0, 64, 64, 200, 256, 256]),
    # documents exactly equal to tiles
    (512, 4, "contiguous", 32, 32, np.arange(0, 513, 32)),
    # one document crossing every chunk
    (1024, 8, "zigzag", 64, 64, [0, 1024]),
    (1024, 8, "contiguous", 64, 16, [0, 1024]),
]


@pytest.mark.parametrize("case", EDGE)
def test_edge_cases(case):
    N, P, layout, bm, bn, cu = case
    for r in range(P):
        _compare(np.asarray(cu, dtype=np.int32), N, P, layout, r, bm, bn)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c5m"])
def test_workload_plans(name):
    w = make_workload(name)
    shards = [w.shard] if w.shard is not None else range(w.sp_degree)
    pairs = []
    for r in shards:
        got = _compare(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, r, w.block_m, w.block_n)
        pairs.append(int(got["useful_pairs"].sum()))
    if w.shard is None:
        # the critical shard is the argmax of useful pairs (ties: lowest id), same as the oracle's count
        ref = oracle.useful_pairs_all_shards(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout)
        assert pairs == ref.tolist()


def test_pair_identity_all_shards():
    # sum over shards and chunks of the planner's pair counts = sum_docs L(L+1)/2
    w = make_workload("c4")
    lengths = np.diff(w.cu_seqlens.astype(np.int64))
    total = sum(int(L.plan(w.cu_seqlens, L.shard_desc(w.total_tokens, w.sp_degree, w.layout, r, 128, 128))
                    ["useful_pairs"].sum()) for r in range(w.sp_degree))
    assert total == int(np.sum(lengths * (lengths + 1) // 2))


def _runs_ok(shard, tiles, sorted_tiles, runs, major, split=0, num_slots=None):
    P = shard.sp_degree
    nq = shard.total_tokens // P // shard.block_m
    covered = np.zeros(len(tiles), dtype=int)
    for slot, t, first, count in runs:
        seg = sorted_tiles[first:first + count]
        if major != L.MAJOR_Q_ALL:
            assert np.all(seg[:, 0] == slot % P)          # a run's tiles belong to its slot's chunk
        assert np.all(seg[:, 1 if major in (L.MAJOR_Q, L.MAJOR_Q_ALL) else 2] == t)
        if split and major == L.MAJOR_Q:
            assert count <= split
        covered[first:first + count] += 1
    assert np.all(covered == 1)
    counts = runs[:, 3]
    assert np.all(np.diff(counts) <= 0)           # longest first
    key = lambda a: sorted(map(tuple, a.tolist()))
    assert key(sorted_tiles) == key(tiles)        # sorted_tiles is a permutation of tiles
    # the documented order of the whole list
    st = ((shard.shard_id - sorted_tiles[:, 0]) % P).astype(np.int64)
    nk = shard.total_tokens // P // shard.block_n
    if major == L.MAJOR_K:
        order = (st * nk + sorted_tiles[:, 2]) * nq + sorted_tiles[:, 1]
        assert np.all(np.diff(order) > 0)
    elif major == L.MAJOR_Q_ALL:
        order = (sorted_tiles[:, 1].astype(np.int64) * P + st) * nk + sorted_tiles[:, 2]
        assert np.all(np.diff(order) > 0)
    else:
        assert np.array_equal(sorted_tiles, tiles)
    if major == L.MAJOR_Q_ALL:
        # one run per q-tile over all chunks, its tiles in ring order
        assert sorted(runs[:, 1].tolist()) == list(range(nq)) and np.all(runs[:, 0] == 0)
        r = shard.shard_id
        for _, t, first, count in runs:
            seg = sorted_tiles[first:first + count]
            assert np.all(seg[:, 1] == t)
            steps = (r - seg[:, 0]) % P
            keys = steps.astype(np.int64) * 100000 + seg[:, 2]
            assert np.all(np.diff(keys) > 0)
        return
    if major == L.MAJOR_Q:
        # every slot in use has exactly one run per q-tile
        slots = sorted(set(runs[:, 0].tolist()))
        assert num_slots == max(slots) + 1
        for s in slots:
            assert sorted(runs[runs[:, 0] == s][:, 1].tolist()) == list(range(nq))
        assert set(s % P for s in slots) == set(tiles[:, 0].tolist())
    else:
        assert np.all(runs[:, 0] == sorted_tiles[runs[:, 2], 0])


@pytest.mark.parametrize("name", ["c2", "c3", "c5m"])
@pytest.mark.parametrize("split", [0, 1, 5])
def test_runs(name, split):
    w = make_workload(name)
    r = w.shard if w.shard is not None else 1
    d = L.shard_desc(w.total_tokens, w.sp_degree, w.layout, r, w.block_m, w.block_n)
    tiles = L.plan(w.cu_seqlens, d)["tiles"]
    for major in (L.MAJOR_Q, L.MAJOR_K, L.MAJOR_Q_ALL):
        sorted_tiles, runs, slots = L.plan_runs(d, tiles, major, split)
        _runs_ok(d, tiles, sorted_tiles, runs, major, split, slots)


def test_split_length():
    d = L.shard_desc(32768, 8, "contiguous", 3, 128, 128)       # 32 k-tiles per chunk
    assert L.split_length(d, 407, 32, 512) == 26                # average 25.4 tiles per workgroup, rounded up
    assert L.split_length(d, 25000, 8, 512) == 0                # every run shorter than the average load
    assert L.split_length(d, 10, 1, 512) == 8                   # floor: a quarter of a chunk's k-tiles
    with pytest.raises(L.HsapError):
        L.split_length(d, 10, 0, 512)


# ---------------------------------------------------------------------------
# block loads of every shard (hsap_load_matrix) and the Q-transfer rebalance (hsap_balance)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(16))
def test_load_matrix_against_oracle(seed):
    rng = np.random.default_rng(2000 + seed)
    P = int(rng.choice([1, 2, 4, 8]))
    layout = str(rng.choice(["contiguous", "zigzag"]))
    bm, bn = int(rng.choice([16, 32, 64])), int(rng.choice([16, 32, 64]))
    split = 2 * P if layout == "zigzag" else P
    N = split * max(bm, bn) * int(rng.integers(1, 3))
    cu = _rand_cu(rng, N)
    tiles, pairs = L.load_matrix(cu, L.shard_desc(N, P, layout, 0, bm, bn))
    ref_tiles, ref_pairs = oracle.load_matrix(cu, N, P, layout, bm, bn)
    assert np.array_equal(tiles, ref_tiles) and np.array_equal(pairs, ref_pairs)


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_load_matrix_workloads(name):
    w = make_workload(name)
    s = L.shard_desc(w.total_tokens, w.sp_degree, w.layout, 0, w.block_m, w.block_n)
    tiles, pairs = L.load_matrix(w.cu_seqlens, s)
    for r in range(w.sp_degree):   # each row is shard r's plan, ring step s at chunk (r - s) mod P
        p = L.plan(w.cu_seqlens, L.shard_desc(w.total_tokens, w.sp_degree, w.layout, r, w.block_m, w.block_n))
        for step in range(w.sp_degree):
            c = (r - step) % w.sp_degree
            assert tiles[r, c] == p["step_offsets"][step + 1] - p["step_offsets"][step]
            assert pairs[r, c] == p["useful_pairs"][step]
    lengths = np.diff(w.cu_seqlens).astype(np.int64)
    assert int(pairs.sum()) == int(np.sum(lengths * (lengths + 1) // 2))


@pytest.mark.parametrize("seed", range(40))
def test_balance_against_oracle(seed):
    rng = np.random.default_rng(3000 + seed)
    P = int(rng.integers(1, 17))
    cost = (rng.integers(0, 50, size=(P, P)) * (rng.random((P, P)) < 0.5)).astype(np.int64)
    if seed % 4 == 0:
        cost[:] = rng.integers(0, 3, size=(P, P))      # many equal costs: the tie rules decide
    exec_rank, load = L.balance(cost)
    ref_exec, ref_load = oracle.q_transfer_balance(cost)
    assert np.array_equal(exec_rank, ref_exec) and np.array_equal(load, ref_load)


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
def test_balance_of_workload_loads(layout):
    w = make_workload("c2")
    tiles, _ = L.load_matrix(w.cu_seqlens, L.shard_desc(w.total_tokens, w.sp_degree, layout, 0, w.block_m,
                                                       w.block_n))
    exec_rank, load = L.balance(tiles)
    ref_exec, ref_load = oracle.q_transfer_balance(tiles)
    assert np.array_equal(exec_rank, ref_exec) and np.array_equal(load, ref_load)
    assert int(load.sum()) == int(tiles.sum())


# ---------------------------------------------------------------------------
# batches of packed sequences
# ---------------------------------------------------------------------------

def _batch_cu(rng, N, B):
    cus = [_rand_cu(rng, N) for _ in range(B)]
    return np.concatenate([cus[0]] + [c[1:] + b * N for b, c in enumerate(cus) if b > 0]).astype(np.int32)


@pytest.mark.parametrize("seed", range(20))
def test_batch_plan_against_oracle(seed):
    rng = np.random.default_rng(4000 + seed)
    P = int(rng.choice([1, 2, 4, 8]))
    B = int(rng.integers(1, 5))
    layout = str(rng.choice(["contiguous", "zigzag"]))
    bm, bn = int(rng.choice([16, 32, 64])), int(rng.choice([16, 32, 64]))
    split = 2 * P if layout == "zigzag" else P
    N = split * max(bm, bn) * int(rng.integers(1, 3))
    cu = _batch_cu(rng, N, B)
    r = int(rng.integers(0, P))
    got = L.plan(cu, L.shard_desc(N, P, layout, r, bm, bn, batch=B))
    ref = oracle.batch_plan_shard(cu, N, B, P, layout, r, bm, bn)
    assert np.array_equal(got["tiles"], ref["tiles"])
    assert np.array_equal(got["step_offsets"], ref["step_offsets"])
    assert np.array_equal(got["useful_pairs"], ref["useful_pairs"])
    tiles, pairs = L.load_matrix(cu, L.shard_desc(N, P, layout, 0, bm, bn, batch=B))
    lengths = np.diff(cu).astype(np.int64)
    assert int(pairs.sum()) == int(np.sum(lengths * (lengths + 1) // 2))


def test_batch_rejects_documents_across_sequences():
    N, P = 256, 2
    s = L.shard_desc(N, P, "contiguous", 0, 32, 32, batch=2)
    with pytest.raises(L.HsapError):
        L.plan(np.array([0, 100, 300, 512], dtype=np.int32), s)     # a document over 256
    with pytest.raises(L.HsapError):
        L.plan(np.array([0, 256], dtype=np.int32), s)                # covers one sequence only
    L.plan(np.array([0, 100, 256, 300, 512], dtype=np.int32), s)
    with pytest.raises(L.HsapError):                                 # B * N beyond 2^31 - 1
        L.plan(np.array([0, 1 << 30], dtype=np.int32), L.shard_desc(1 << 30, 1, "contiguous", 0, 64, 64, batch=2))
