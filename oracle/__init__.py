"""fp64 CPU oracle for document-masked packed causal attention on one sequence-parallel shard.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or run
anything in this package: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP library
(no kernels, headers, helpers, tables or constant generators) and imports
nothing from it.

What it computes, with the passages it follows (HSAP paper, arxiv 2606.30460):

* ``attention.doc_starts``/``attention.allowed`` -- the packed-sequence mask:
  attention only within each document of the packed sequence (the
  sequence-packing section, where the cumulative-length array confines
  attention to each segment), causal inside a document so that it matches the
  behaviour of causal attention on each document alone.
* ``attention.attention_fwd`` -- scaled dot-product attention,
  Softmax(QK^T / sqrt(d)) V per head (the attention equation of the
  inter-group sequence-parallelism section), restricted to the allowed pairs;
  also returns the log-sum-exp of every row.
* ``attention.lse_merge`` -- the online-softmax combination of partial results
  that a ring rank accumulates as K/V chunks arrive (same section; the
  combination is the one of Milakov and Gimelshein that the paper cites).
* ``attention.attention_bwd`` -- gradients of the same function, taken from
  its definition (the paper's per-rank code moves dq, dkv and do tensors in the
  backward pass, instruction table of the SAP section).
* ``layout.shard_positions`` -- which global tokens a shard holds: contiguous
  slices along the length (inter-group SP and the HSAP hierarchy sections) or
  the zigzag split used for ring load balance (the paper defers to LightSeq's
  balancing in the compile-algorithm section).
* ``plan`` -- the per-shard tile classification that the compile step's block
  partition performs (compile step 1 of the SAP section), at tile granularity.
* ``balance`` -- the per-(shard, chunk) block sizes of every shard and the
  Q-transfer rebalance of the blocks over ranks (compile step 2, and the
  balancing of InterSP groups by transferring Q blocks).
* ``batch`` -- batches of packed sequences (each sharded the same way, never
  attending across sequences), computed one sequence at a time.
* ``fp8`` -- the e4m3 quantisation of Q and K for the fp8 score variant (an
  extension beyond the paper's bf16 attention; its attention is the oracle's
  attention on the dequantised values).
* ``schedule`` -- the per-rank instruction lists of the forward and backward
  passes (the jitted code generation of the SAP section, with the paper's
  instruction set: q, kv, o, dq, dkv, do messages), arranged in stages with
  matched sends and receives.

Parity status: every function above is pinned by ``tests/test_oracle_pins.py``
against brute force, closed forms, library routines or invariants; none is
"parity unpinned".
"""
from .attention import (  # noqa: F401
    allowed_mask_dense,
    attention_bwd,
    attention_fwd,
    doc_starts,
    lse_merge,
    shard_backward,
    shard_forward,
)
from .layout import ring_chunk, shard_positions  # noqa: F401
from .plan import (  # noqa: F401
    plan_shard,
    tile_pair_counts,
    tile_pair_counts_bruteforce,
    useful_pairs_all_shards,
)
from .balance import load_matrix, q_transfer_balance  # noqa: F401
from .schedule import backward_program, forward_program  # noqa: F401
from .batch import batch_plan_shard, batch_shard_backward, batch_shard_forward, split_batch  # noqa: F401
from .fp8 import decode_fp8, dequantize_fp8, quantize_fp8  # noqa: F401
