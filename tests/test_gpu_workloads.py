"""The benchmark's workloads at full size, every row, against the fp64 oracle.

Each workload runs twice on the GPU on the same seeded inputs:

* through the step executor as the benchmark times it (host plan and one upload,
  document starts found in cu_seqlens, the partial forward with final-slot writes
  of single-part q-tiles, the merge of the listed q-tiles, the two-stage form of
  the forward, and for the forward+backward workloads the backward with delta
  folded into the dQ kernel and bf16 gradients), plus the fused forward from the
  same plan (the benchmark times it with an executor of its own; its lists are
  the same);
* through the entry points one by one (per-position document starts, every
  partial slot kept, fp32 gradient accumulators), whose partials are compared
  chunk by chunk.

Every output is pre-filled with NaN, so a row the GPU path leaves unwritten fails.
Bars: O max-abs <= 2e-2, LSE max-abs <= 1e-3, the set of -inf rows of every
partial identical, gradients max|g - ref| / max|ref| <= 3e-2; the executor's bf16
gradients equal the entry points' fp32 gradients rounded to bf16, bit for bit.

For the 131072- and 262144-token workloads the backward is compared with the
oracle on two K/V heads (with their query heads) and on every row, with the
workloads' 128-row q-tiles and again with 256-row q-tiles (the eight-wave
forward and dQ kernels); the other heads are held to the entry-point path bit
for bit.
"""
import sys
import time

import numpy as np
import pytest
import torch

from _harness import GRAD_RTOL, LSE_ATOL, O_ATOL, Case, compare_backward, compare_forward, max_abs, rel_max
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16).float().numpy()


def _no_nan(out, keys):
    for key in keys:
        assert not np.isnan(out[key]).any(), "%s has rows the GPU path did not write" % key


def _executor_forward_report(ex, ref, heads=None):
    hs = slice(None) if heads is None else heads
    rep = {}
    for tag in ("", "_fused", "_staged"):
        o, lse = ex["o" + tag][:, hs], ex["lse" + tag][hs]
        rep["o" + tag] = max_abs(o, ref["o"])
        rep["lse" + tag] = max_abs(lse, ref["lse"])
        assert rep["o" + tag] <= O_ATOL and rep["lse" + tag] <= LSE_ATOL, rep
    # the two-stage form launches the same kernels over the same lists
    assert np.array_equal(ex["o_staged"], ex["o"]) and np.array_equal(ex["lse_staged"], ex["lse"])
    return rep


@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
def test_workload_forward_every_row(name):
    w = make_workload(name)
    c = Case.from_workload(w)
    _say("workload", name, "shard", c.shard, "rows", w.total_tokens // w.sp_degree)
    t0 = time.perf_counter()
    ref = c.run_oracle()
    _say("oracle %.1f s" % (time.perf_counter() - t0))
    ex = c.run_executor()
    _no_nan(ex, ("o", "lse", "o_fused", "lse_fused", "o_staged", "lse_staged"))
    rep = _executor_forward_report(ex, ref)
    _say(name, "executor", {k: round(v, 6) for k, v in rep.items()}, ex["info"])
    del ex
    gpu = c.run_gpu()
    _no_nan(gpu, ("o", "lse", "o_fused", "lse_fused"))
    rep = compare_forward(gpu, ref)
    _say(name, "entry points", {k: round(v, 6) for k, v in rep.items() if not k.startswith(("o_part", "lse_part"))})


def _backward_case(name, block_m=None):
    w = make_workload(name)
    c = Case.from_workload(w)
    bm = w.block_m if block_m is None else block_m
    if not c.backward or bm != w.block_m:  # a forward workload run forward + backward, or other q-tiles
        c = Case(w.cu_seqlens, w.total_tokens, w.sp_degree, w.layout, c.shard, w.heads_q, w.heads_kv, w.head_dim,
                 bm, w.block_n, w.seed, backward=True)
    return w, c


@pytest.mark.parametrize("name", ["c5", "c5m"])
def test_workload_backward_every_row(name):
    w, c = _backward_case(name)
    _say("workload", name, "shard", c.shard)
    t0 = time.perf_counter()
    ref = c.run_oracle()
    _say("oracle %.1f s" % (time.perf_counter() - t0))
    ex = c.run_executor()
    _no_nan(ex, ("o", "lse", "o_fused", "lse_fused", "dq", "dk", "dv"))
    rep = _executor_forward_report(ex, ref["fwd"])
    rep.update(compare_backward(ex, ref))
    _say(name, "executor", {k: round(v, 6) for k, v in rep.items()})
    gpu = c.run_gpu()
    compare_forward(gpu, ref["fwd"])
    _say(name, "entry points", compare_backward(gpu, ref))
    assert np.array_equal(ex["dq"], gpu["dq_bf16"])
    assert np.array_equal(ex["dk"], _bf16(gpu["dk"])) and np.array_equal(ex["dv"], _bf16(gpu["dv"]))


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_workload_backward_long_documents(name):
    """The long-document workloads forward + backward from one executor, with their own q-tiles (128
    rows) and with 256-row q-tiles; the oracle (independent of the tiling) is computed once."""
    w = make_workload(name)
    kv = [0, w.heads_kv - 1]
    ref = None
    for bm in (w.block_m, 256):
        _, c = _backward_case(name, block_m=bm)
        hs = c.q_heads(kv)
        _say("workload", name, "fwd+bwd, BM", bm, "shard", c.shard, "oracle on K/V heads", kv)
        ex = c.run_executor()
        _no_nan(ex, ("o", "lse", "dq", "dk", "dv"))
        gpu = c.run_gpu()
        # every head: the executor's bf16 gradients are the entry points' fp32 ones rounded
        assert np.array_equal(ex["dq"], gpu["dq_bf16"])
        assert np.array_equal(ex["dk"], _bf16(gpu["dk"])) and np.array_equal(ex["dv"], _bf16(gpu["dv"]))
        del gpu
        if ref is None:
            t0 = time.perf_counter()
            ref = c.run_oracle(kv_heads=kv)
            _say("oracle %.1f s" % (time.perf_counter() - t0))
        rep = _executor_forward_report(ex, ref["fwd"], heads=hs)
        rep.update(dq=rel_max(ex["dq"][:, hs], ref["dq"]), dk=rel_max(ex["dk"][:, :, kv], ref["dk"]),
                   dv=rel_max(ex["dv"][:, :, kv], ref["dv"]))
        _say(name, "BM", bm, {k: round(v, 6) for k, v in rep.items()}, ex["info"])
        assert max(rep["dq"], rep["dk"], rep["dv"]) <= GRAD_RTOL, rep
        del ex


@pytest.mark.parametrize("name", ["c2", "c5", "c5m"])
def test_workload_tile_list_entry_points(name):
    """The boundary's tile-list calls (hsap_partial_attn_fwd / _bwd once per ring step on that chunk's
    tiles from hsap_plan) on the 32768-token workloads, every row: each chunk's partial, the merge and,
    for the forward + backward workloads, the gradients against the oracle."""
    from _harness import compare_tile_list
    w = make_workload(name)
    c = Case.from_workload(w)
    _say("workload", name, "tile-list calls, shard", c.shard)
    got = c.run_tile_list()
    ref = c.run_oracle()
    rep = compare_tile_list(got, ref["fwd"] if c.backward else ref)
    if c.backward:
        rep.update(compare_backward(got, ref))
    _say(name, {k: round(v, 6) for k, v in rep.items() if not k.startswith(("o_part", "lse_part"))})
