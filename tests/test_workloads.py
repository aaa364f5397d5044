"""The synthetic input generators: determinism and the stated length distributions."""
import numpy as np
import pytest

from workloads import (CONFIGS, cu_seqlens_from_lengths, doc_lengths_extreme, doc_lengths_lognormal,
                       doc_lengths_mixed, doc_lengths_pareto, doc_lengths_uniform_partition, make_workload,
                       random_bf16)


def test_uniform_partition_seed0():
    # 5 cut points iid uniform in 0..2048-96 (inclusive), sorted; gaps + 16
    assert doc_lengths_uniform_partition(2048, 6, 16, 0) == [542, 91, 413, 261, 434, 307]


@pytest.mark.parametrize("name", list(CONFIGS))
def test_workloads_cover_total(name):
    w = make_workload(name)
    assert sum(w.lengths) == w.total_tokens * w.batch
    assert all(x > 0 for x in w.lengths)
    cu = w.cu_seqlens
    assert cu.dtype == np.int32 and cu[0] == 0 and cu[-1] == w.total_tokens * w.batch
    assert all(b * w.total_tokens in cu for b in range(w.batch))   # every sequence starts a document
    assert w.total_tokens % (w.sp_degree * (2 if w.layout == "zigzag" else 1)) == 0
    n = w.total_tokens // w.sp_degree
    assert n % w.block_m == 0 and n % w.block_n == 0
    assert make_workload(name).lengths == w.lengths          # deterministic


def test_distribution_bounds():
    ln = doc_lengths_lognormal(32768, 2048, 1.0, 128, 16384, 0)
    assert all(128 <= x <= 16384 for x in ln[:-1])
    mx = doc_lengths_mixed(131072, 0.1, (64, 512), (8192, 65536), 0)
    assert all((64 <= x <= 512) or (8192 <= x <= 65536) for x in mx[:-1])
    pa = doc_lengths_pareto(262144, 1.2, 32, 131072, 0)
    assert all(32 <= x <= 131072 for x in pa)
    ex = doc_lengths_extreme(32768, 30000, 8, True)
    assert ex[0] == 30000 and len(ex) == 347 and set(ex[1:]) == {8}
    assert doc_lengths_extreme(32768, 30000, 8, False)[-1] == 30000


def test_random_bf16_seeded():
    a = random_bf16((4, 3), 5)
    b = random_bf16((4, 3), 5)
    assert a.dtype.is_floating_point and str(a.dtype) == "torch.bfloat16"
    assert bool((a == b).all())
    assert not bool((a == random_bf16((4, 3), 6)).all())


def test_cu_seqlens():
    assert cu_seqlens_from_lengths([3, 0, 5]).tolist() == [0, 3, 3, 8]
