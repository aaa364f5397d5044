"""Per-rank instruction lists of the forward pass (hsap_emit_forward) against the oracle's emitter,
bit for bit, and the lists themselves against what they must do.

Structural checks: every send has the matching receive at the same stage of the peer's list and
the other way round; every non-empty block is computed once, on its assigned rank, from inputs
received at an earlier stage and not overwritten since; within a stage no slot is both read by
a transfer and written by the computation (or written by a receive and read by the computation);
each shard merges all its parts after the last of them arrived.  End to end: the lists executed
on fp64 data, each computing op through the oracle's attention and each merge through its LSE
merge, give every shard the oracle's result for that shard.
"""
from collections import defaultdict

import numpy as np
import pytest

import oracle
from oracle.schedule import OP_COMPUTE, OP_MERGE, OP_RECV, OP_SEND, T_KV, T_O, T_Q
from paper_2606_30460_amd import _lib as L
from workloads import make_workload


def _as_tuples(ops):
    return [tuple(int(x) for x in o) for o in ops]


def _random_case(rng):
    P = int(rng.integers(1, 9))
    tiles = rng.integers(0, 30, size=(P, P)) * (rng.random((P, P)) < 0.6)
    if rng.random() < 0.8:
        np.fill_diagonal(tiles, rng.integers(1, 30, size=P))     # real plans always have the diagonal
    ex = np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
    move = rng.random((P, P)) < 0.4
    ex[move] = np.broadcast_to(np.arange(P, dtype=np.int32)[None, :], (P, P))[move]
    return tiles.astype(np.int64), ex


@pytest.mark.parametrize("seed", range(40))
def test_emit_matches_oracle(seed):
    tiles, ex = _random_case(np.random.default_rng(500 + seed))
    ops, stages = L.emit_forward(tiles, ex)
    ref, ref_stages = oracle.forward_program(tiles, ex)
    assert stages == ref_stages
    assert [_as_tuples(o) for o in ops] == ref


def _check_structure(prog, tiles, ex):
    P = tiles.shape[0]
    sends, recvs = defaultdict(int), defaultdict(int)
    computed = defaultdict(int)
    parts = [[c for c in range(P) if tiles[r, c] > 0] for r in range(P)]
    for e, ops in enumerate(prog):
        stages = [o[3] for o in ops]
        assert stages == sorted(stages)
        recv_slot = {}          # (tensor, slot) -> (what, stage received)
        result_slot = {}        # slot -> ((shard, chunk), stage computed)
        part_arrived = {}       # part index -> stage
        by_stage = defaultdict(list)
        for o in ops:
            by_stage[o[3]].append(o)
        for t in sorted(by_stage):
            read_now, written_now = set(), set()
            for o in by_stage[t]:
                op, tensor, peer, _, shard, chunk, in_slot, out_slot = o
                if op == OP_SEND:
                    sends[(e, peer, t, tensor, shard, chunk)] += 1
                    if tensor == T_O:
                        assert result_slot[in_slot][0] == (shard, chunk) and result_slot[in_slot][1] < t
                        read_now.add(("result", in_slot))
                    elif tensor == T_Q:
                        assert shard == e and in_slot == -1
                    else:
                        assert chunk == e and in_slot == -1
                elif op == OP_RECV:
                    recvs[(peer, e, t, tensor, shard, chunk)] += 1
                    if tensor == T_O:
                        assert shard == e and out_slot == parts[e].index(chunk)
                        part_arrived[out_slot] = t
                    else:
                        recv_slot[(tensor, out_slot)] = ((shard if tensor == T_Q else chunk), t)
                        written_now.add((tensor, out_slot))
                elif op == OP_COMPUTE:
                    computed[(shard, chunk)] += 1
                    assert ex[shard, chunk] == e and tiles[shard, chunk] > 0
                    if shard != e:        # Q from slot in_slot, received earlier
                        assert recv_slot[(T_Q, in_slot)] [0] == shard and recv_slot[(T_Q, in_slot)][1] < t
                        read_now.add((T_Q, in_slot))
                        result_slot[out_slot] = ((shard, chunk), t)
                        written_now.add(("result", out_slot))
                    else:
                        if chunk != e:
                            assert recv_slot[(T_KV, in_slot)][0] == chunk and recv_slot[(T_KV, in_slot)][1] < t
                            read_now.add((T_KV, in_slot))
                        else:
                            assert in_slot == -1
                        assert out_slot == parts[e].index(chunk)
                        part_arrived[out_slot] = t
                else:
                    assert op == OP_MERGE and shard == e and out_slot == len(parts[e])
                    assert sorted(part_arrived) == list(range(len(parts[e])))
                    assert max(part_arrived.values()) <= t
            assert not (read_now & written_now), (e, t, read_now & written_now)
    assert sends == recvs
    assert all(v == 1 for v in sends.values())
    for r in range(P):
        for c in range(P):
            assert computed[(r, c)] == (1 if tiles[r, c] > 0 else 0)


@pytest.mark.parametrize("seed", range(40))
def test_program_structure_random(seed):
    tiles, ex = _random_case(np.random.default_rng(700 + seed))
    prog, _ = oracle.forward_program(tiles, ex)
    _check_structure(prog, tiles, ex)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
@pytest.mark.parametrize("balanced", [False, True])
def test_program_structure_workloads(name, balanced):
    w = make_workload(name)
    tiles, _ = L.load_matrix(w.cu_seqlens, L.shard_desc(w.total_tokens, w.sp_degree, w.layout, 0, w.block_m,
                                                       w.block_n))
    P = w.sp_degree
    ex = L.balance(tiles)[0] if balanced else np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
    ops, stages = L.emit_forward(tiles, ex)
    prog = [_as_tuples(o) for o in ops]
    assert (prog, stages) == oracle.forward_program(tiles, ex)
    _check_structure(prog, tiles, ex)


def _execute(prog, stages, q, k, v, cu, N, P, layout):
    """Run the lists on fp64 data: every rank's buffers, stage by stage (transfers, then computation,
    then the merge), each block through the oracle's attention."""
    pos = [oracle.shard_positions(N, P, layout, x) for x in range(P)]
    own_q = [q[pos[x]] for x in range(P)]
    own_kv = [(k[pos[x]], v[pos[x]]) for x in range(P)]
    recv = [dict() for _ in range(P)]
    result = [dict() for _ in range(P)]
    part = [dict() for _ in range(P)]
    out = [None] * P
    for t in range(stages):
        snapshot = [dict(result[e]) for e in range(P)]      # what the stage's sends read
        for e in range(P):
            for o in prog[e]:
                op, tensor, peer, st, shard, chunk, in_slot, out_slot = o
                if st != t or op != OP_RECV:
                    continue
                if tensor == T_Q:
                    recv[e][(T_Q, out_slot)] = own_q[peer]
                elif tensor == T_KV:
                    recv[e][(T_KV, out_slot)] = own_kv[peer]
                else:
                    send = [s for s in prog[peer] if s[0] == OP_SEND and s[3] == t and s[2] == e and s[1] == T_O
                            and s[4] == shard and s[5] == chunk]
                    part[e][out_slot] = snapshot[peer][send[0][6]]
        for e in range(P):
            for o in prog[e]:
                op, tensor, peer, st, shard, chunk, in_slot, out_slot = o
                if st != t:
                    continue
                if op == OP_COMPUTE:
                    qq = own_q[e] if shard == e else recv[e][(T_Q, in_slot)]
                    kk, vv = own_kv[e] if chunk == e else recv[e][(T_KV, in_slot)]
                    res = oracle.attention_fwd(qq, kk, vv, pos[shard], pos[chunk], cu)
                    if shard == e:
                        part[e][out_slot] = res
                    else:
                        result[e][out_slot] = res
                elif op == OP_MERGE:
                    out[e] = oracle.lse_merge([part[e][i][0] for i in range(out_slot)],
                                              [part[e][i][1] for i in range(out_slot)])
    return out


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("seed", range(3))
def test_program_runs_to_oracle_result(layout, seed):
    rng = np.random.default_rng(40 + seed)
    P, H, d, bm, bn = 4, 2, 8, 8, 8
    N = 2 * P * 16
    cu = np.array([0, N]) if seed == 0 else np.sort(np.concatenate([[0, N], rng.integers(0, N + 1, size=5)]))
    q, k, v = (rng.standard_normal((N, H, d)) for _ in range(3))
    tiles, _ = oracle.load_matrix(cu, N, P, layout, bm, bn)
    for ex in (np.repeat(np.arange(P)[:, None], P, axis=1), oracle.q_transfer_balance(tiles)[0]):
        prog, stages = oracle.forward_program(tiles, ex)
        out = _execute(prog, stages, q, k, v, cu, N, P, layout)
        for r in range(P):
            ref = oracle.shard_forward(q, k, v, cu, N, P, layout, r)
            assert np.max(np.abs(out[r][0] - ref["o"])) <= 1e-12
            assert np.array_equal(np.isneginf(out[r][1]), np.isneginf(ref["lse"]))
            assert np.max(np.abs(out[r][1] - ref["lse"])) <= 1e-12


def test_emit_validates():
    tiles = np.ones((2, 2), dtype=np.int64)
    L.emit_forward(tiles, np.array([[0, 1], [0, 1]], dtype=np.int32))     # off-diagonal blocks on their chunk's rank
    with pytest.raises(L.HsapError):                                      # diagonal block (1, 1) on rank 0
        L.emit_forward(tiles, np.array([[0, 0], [1, 0]], dtype=np.int32))
    ex3 = np.repeat(np.arange(3, dtype=np.int32)[:, None], 3, axis=1)
    ex3[1, 2] = 0                                                         # block (1, 2) on rank 0: neither 1 nor 2
    with pytest.raises(L.HsapError):
        L.emit_forward(np.ones((3, 3), dtype=np.int64), ex3)
    empty = np.ones((3, 3), dtype=np.int64)
    empty[1, 2] = 0                                                       # an empty block's rank is not read
    L.emit_forward(empty, ex3)
    with pytest.raises(L.HsapError):
        L.emit_forward(-tiles, np.zeros((2, 2), dtype=np.int32))


# ---------------------------------------------------------------------------
# backward program (dq, dkv, do messages)
# ---------------------------------------------------------------------------

from oracle.schedule import T_DKV, T_DO, T_DQ  # noqa: E402


@pytest.mark.parametrize("seed", range(40))
def test_emit_backward_matches_oracle(seed):
    tiles, ex = _random_case(np.random.default_rng(900 + seed))
    ops, stages = L.emit_backward(tiles, ex)
    ref, ref_stages = oracle.backward_program(tiles, ex)
    assert stages == ref_stages
    assert [_as_tuples(o) for o in ops] == ref
    # the backward computes every block at its forward stage, on its forward rank
    fwd, fwd_stages = oracle.forward_program(tiles, ex)
    assert fwd_stages == stages
    for e in range(tiles.shape[0]):
        assert [(o[3], o[4], o[5]) for o in ref[e] if o[0] == OP_COMPUTE] == \
            [(o[3], o[4], o[5]) for o in fwd[e] if o[0] == OP_COMPUTE]


def _check_backward_structure(prog, tiles, ex):
    P = tiles.shape[0]
    sends, recvs = defaultdict(int), defaultdict(int)
    computed = defaultdict(int)
    dq_parts = [[c for c in range(P) if tiles[r, c] > 0] for r in range(P)]
    dkv_parts = [[r for r in range(P) if tiles[r, c] > 0] for c in range(P)]
    for e, ops in enumerate(prog):
        stages = [o[3] for o in ops]
        assert stages == sorted(stages)
        recv_slot = {}          # (tensor, slot) -> (shard or chunk held, stage received)
        result_slot = {}        # slot -> (tensor, (shard, chunk), stage computed)
        dq_arrived, dkv_arrived = {}, {}
        by_stage = defaultdict(list)
        for o in ops:
            by_stage[o[3]].append(o)
        for t in sorted(by_stage):
            read_now, written_now = set(), set()
            for o in by_stage[t]:
                op, tensor, peer, _, shard, chunk, in_slot, out_slot = o
                if op == OP_SEND:
                    sends[(e, peer, t, tensor, shard, chunk)] += 1
                    if tensor in (T_DQ, T_DKV):
                        assert result_slot[in_slot][:2] == (tensor, (shard, chunk)) and result_slot[in_slot][2] < t
                        read_now.add(("result", in_slot))
                    elif tensor in (T_Q, T_DO):
                        assert shard == e and in_slot == -1
                    else:
                        assert tensor == T_KV and chunk == e and in_slot == -1
                elif op == OP_RECV:
                    recvs[(peer, e, t, tensor, shard, chunk)] += 1
                    if tensor == T_DQ:
                        assert shard == e and out_slot == dq_parts[e].index(chunk) and out_slot not in dq_arrived
                        dq_arrived[out_slot] = t
                    elif tensor == T_DKV:
                        assert chunk == e and out_slot == dkv_parts[e].index(shard) and out_slot not in dkv_arrived
                        dkv_arrived[out_slot] = t
                    else:
                        recv_slot[(tensor, out_slot)] = ((chunk if tensor == T_KV else shard), t)
                        written_now.add((tensor, out_slot))
                elif op == OP_COMPUTE:
                    computed[(shard, chunk)] += 1
                    assert ex[shard, chunk] == e and tiles[shard, chunk] > 0
                    if shard == chunk:
                        assert in_slot == -1 and out_slot == -1
                    if shard != e:        # Q and dO from slot in_slot; dQ leaves through result slot out_slot
                        for tensor_in in (T_Q, T_DO):
                            assert recv_slot[(tensor_in, in_slot)][0] == shard
                            assert recv_slot[(tensor_in, in_slot)][1] < t
                            read_now.add((tensor_in, in_slot))
                        result_slot[out_slot] = (T_DQ, (shard, chunk), t)
                        written_now.add(("result", out_slot))
                    else:
                        dq_arrived[dq_parts[e].index(chunk)] = t
                    if chunk != e:        # K/V from slot in_slot; dK/dV leave through result slot out_slot
                        assert recv_slot[(T_KV, in_slot)][0] == chunk and recv_slot[(T_KV, in_slot)][1] < t
                        read_now.add((T_KV, in_slot))
                        result_slot[out_slot] = (T_DKV, (shard, chunk), t)
                        written_now.add(("result", out_slot))
                    else:
                        dkv_arrived[dkv_parts[e].index(shard)] = t
                else:
                    assert op == OP_MERGE
                    if tensor == T_DQ:
                        assert shard == e and out_slot == len(dq_parts[e])
                        assert sorted(dq_arrived) == list(range(len(dq_parts[e])))
                        assert max(dq_arrived.values()) <= t
                    else:
                        assert tensor == T_DKV and chunk == e and out_slot == len(dkv_parts[e])
                        assert sorted(dkv_arrived) == list(range(len(dkv_parts[e])))
                        assert max(dkv_arrived.values()) <= t
            assert not (read_now & written_now), (e, t, read_now & written_now)
        assert (len(dq_parts[e]) > 0) == any(o[0] == OP_MERGE and o[1] == T_DQ for o in ops)
        assert (len(dkv_parts[e]) > 0) == any(o[0] == OP_MERGE and o[1] == T_DKV for o in ops)
    assert sends == recvs
    assert all(v == 1 for v in sends.values())
    for r in range(P):
        for c in range(P):
            assert computed[(r, c)] == (1 if tiles[r, c] > 0 else 0)


@pytest.mark.parametrize("seed", range(40))
def test_backward_program_structure_random(seed):
    tiles, ex = _random_case(np.random.default_rng(1100 + seed))
    prog, _ = oracle.backward_program(tiles, ex)
    _check_backward_structure(prog, tiles, ex)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
@pytest.mark.parametrize("balanced", [False, True])
def test_backward_program_structure_workloads(name, balanced):
    w = make_workload(name)
    tiles, _ = L.load_matrix(w.cu_seqlens, L.shard_desc(w.total_tokens, w.sp_degree, w.layout, 0, w.block_m,
                                                       w.block_n))
    P = w.sp_degree
    ex = L.balance(tiles)[0] if balanced else np.repeat(np.arange(P, dtype=np.int32)[:, None], P, axis=1)
    ops, stages = L.emit_backward(tiles, ex)
    prog = [_as_tuples(o) for o in ops]
    assert (prog, stages) == oracle.backward_program(tiles, ex)
    _check_backward_structure(prog, tiles, ex)


def _execute_backward(prog, stages, tiles, q, k, v, d_o, cu, N, P, layout):
    """Run the backward lists on fp64 data.  Every rank starts from its own Q, K/V, dO and its
    shard's final LSE and delta (from the oracle's forward); each computing op goes through the
    oracle's attention backward, each merge sums the parts in index order."""
    pos = [oracle.shard_positions(N, P, layout, x) for x in range(P)]
    dq_parts = [[c for c in range(P) if tiles[r, c] > 0] for r in range(P)]
    dkv_parts = [[r for r in range(P) if tiles[r, c] > 0] for c in range(P)]
    own_q = [q[pos[x]] for x in range(P)]
    own_kv = [(k[pos[x]], v[pos[x]]) for x in range(P)]
    own_do = []
    for x in range(P):
        f = oracle.shard_forward(q, k, v, cu, N, P, layout, x)
        dos = d_o[pos[x]]
        own_do.append((dos, f["lse"], np.einsum("nhd,nhd->hn", dos, f["o"])))
    recv = [dict() for _ in range(P)]
    result = [dict() for _ in range(P)]
    dq_part, dkv_part = [dict() for _ in range(P)], [dict() for _ in range(P)]
    dq, dk, dv = [None] * P, [None] * P, [None] * P
    for t in range(stages):
        snapshot = [dict(result[e]) for e in range(P)]      # what the stage's sends read
        for e in range(P):
            for o in prog[e]:
                op, tensor, peer, st, shard, chunk, in_slot, out_slot = o
                if st != t or op != OP_RECV:
                    continue
                if tensor == T_Q:
                    recv[e][(T_Q, out_slot)] = own_q[peer]
                elif tensor == T_DO:
                    recv[e][(T_DO, out_slot)] = own_do[peer]
                elif tensor == T_KV:
                    recv[e][(T_KV, out_slot)] = own_kv[peer]
                else:
                    send = [s for s in prog[peer] if s[0] == OP_SEND and s[3] == t and s[2] == e and s[1] == tensor
                            and s[4] == shard and s[5] == chunk]
                    (dq_part if tensor == T_DQ else dkv_part)[e][out_slot] = snapshot[peer][send[0][6]]
        for e in range(P):
            for o in prog[e]:
                op, tensor, peer, st, shard, chunk, in_slot, out_slot = o
                if st != t:
                    continue
                if op == OP_COMPUTE:
                    qq = own_q[e] if shard == e else recv[e][(T_Q, in_slot)]
                    dos, lse, delta = own_do[e] if shard == e else recv[e][(T_DO, in_slot)]
                    kk, vv = own_kv[e] if chunk == e else recv[e][(T_KV, in_slot)]
                    g_q, g_k, g_v = oracle.attention_bwd(qq, kk, vv, dos, lse, delta, pos[shard], pos[chunk], cu)
                    if shard == e:
                        dq_part[e][dq_parts[e].index(chunk)] = g_q
                    else:
                        result[e][out_slot] = g_q
                    if chunk == e:
                        dkv_part[e][dkv_parts[e].index(shard)] = (g_k, g_v)
                    else:
                        result[e][out_slot] = (g_k, g_v)
                elif op == OP_MERGE and tensor == T_DQ:
                    dq[e] = sum(dq_part[e][i] for i in range(out_slot))
                elif op == OP_MERGE:
                    dk[e] = sum(dkv_part[e][i][0] for i in range(out_slot))
                    dv[e] = sum(dkv_part[e][i][1] for i in range(out_slot))
    return dq, dk, dv


@pytest.mark.parametrize("layout", ["contiguous", "zigzag"])
@pytest.mark.parametrize("seed", range(3))
def test_backward_program_runs_to_oracle_gradients(layout, seed):
    """Each shard's dQ and each chunk's dK/dV, summed over every shard's contribution, equal the
    oracle's shard backward, for the ring and the balanced assignment (GQA, two K/V heads)."""
    rng = np.random.default_rng(60 + seed)
    P, hq, hkv, d, bm, bn = 4, 4, 2, 8, 8, 8
    N = 2 * P * 16
    cu = np.array([0, N]) if seed == 0 else np.sort(np.concatenate([[0, N], rng.integers(0, N + 1, size=5)]))
    q, d_o = rng.standard_normal((N, hq, d)), rng.standard_normal((N, hq, d))
    k, v = rng.standard_normal((N, hkv, d)), rng.standard_normal((N, hkv, d))
    tiles, _ = oracle.load_matrix(cu, N, P, layout, bm, bn)
    refs = [oracle.shard_backward(q, k, v, d_o, cu, N, P, layout, r) for r in range(P)]
    for ex in (np.repeat(np.arange(P)[:, None], P, axis=1), oracle.q_transfer_balance(tiles)[0]):
        prog, stages = oracle.backward_program(tiles, ex)
        dq, dk, dv = _execute_backward(prog, stages, tiles, q, k, v, d_o, cu, N, P, layout)
        for x in range(P):
            assert np.max(np.abs(dq[x] - refs[x]["dq"])) <= 1e-12
            assert np.max(np.abs(dk[x] - sum(refs[r]["dk"][x] for r in range(P)))) <= 1e-12
            assert np.max(np.abs(dv[x] - sum(refs[r]["dv"][x] for r in range(P)))) <= 1e-12


def test_emit_backward_validates():
    tiles = np.ones((2, 2), dtype=np.int64)
    with pytest.raises(L.HsapError):                                      # diagonal block (1, 1) on rank 0
        L.emit_backward(tiles, np.array([[0, 0], [1, 0]], dtype=np.int32))
    with pytest.raises(L.HsapError):
        L.emit_backward(-tiles, np.zeros((2, 2), dtype=np.int32))
