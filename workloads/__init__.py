"""Seeded synthetic inputs for document-masked packed attention.

This module only draws numbers: document lengths of packed sequences and
random Q/K/V/dO tensors.  It holds none of the attention method's arithmetic
(no masks, no shard layouts, no softmax), so both the fp64 oracle's tests and
the GPU path's harness can take their inputs from it without sharing any of
the method between them.

The paper packs unrelated documents into one long sequence and describes each
packed batch by its cumulative document lengths (the ``cu_len`` array of the
sequence-packing section).  The paper's own datasets are not available, so the
samplers below stand in for them with the length distributions listed in
``CONFIGS``.
"""
from .synth import (  # noqa: F401
    CONFIGS,
    Workload,
    cu_seqlens_from_lengths,
    doc_lengths_extreme,
    doc_lengths_lognormal,
    doc_lengths_mixed,
    doc_lengths_pareto,
    doc_lengths_uniform_partition,
    make_workload,
    random_bf16,
)
