"""The test harness's head-parallel driver of the oracle (CPU): splitting the oracle's work by
K/V head over host threads and concatenating must reproduce one oracle call on all heads."""
import numpy as np

import oracle
from _harness import oracle_by_kv_heads
from workloads import random_bf16


def test_split_by_kv_heads_equals_one_call():
    N, P, layout, r = 256, 2, "zigzag", 1
    hq, hkv, d = 6, 3, 16
    cu = np.array([0, 40, 41, 130, 256], dtype=np.int32)
    q, k, v, do = (random_bf16((N, h, d), s).float().numpy() for s, h in ((1, hq), (2, hkv), (3, hkv), (4, hq)))
    ref = oracle.shard_forward(q, k, v, cu, N, P, layout, r)
    got = oracle_by_kv_heads(q, k, v, None, cu, N, P, layout, r, list(range(hkv)))
    np.testing.assert_allclose(got["o"], ref["o"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["lse"], ref["lse"], rtol=0, atol=1e-12)
    for a, b in zip(got["lse_parts"], ref["lse_parts"]):
        assert np.array_equal(np.isneginf(a), np.isneginf(b))
    rows = np.array([3, 70, 127])
    sub = oracle_by_kv_heads(q, k, v, None, cu, N, P, layout, r, [2], rows=rows)
    np.testing.assert_allclose(sub["o"], ref["o"][rows][:, 4:6], rtol=0, atol=1e-12)
    refb = oracle.shard_backward(q, k, v, do, cu, N, P, layout, r)
    gotb = oracle_by_kv_heads(q, k, v, do, cu, N, P, layout, r, [0, 2])
    np.testing.assert_allclose(gotb["dq"], refb["dq"][:, [0, 1, 4, 5]], rtol=0, atol=1e-12)
    np.testing.assert_allclose(gotb["dk"], refb["dk"][:, :, [0, 2]], rtol=0, atol=1e-12)
    np.testing.assert_allclose(gotb["dv"], refb["dv"][:, :, [0, 2]], rtol=0, atol=1e-12)
