"""MI355X-native document-masked packed attention for one sequence-parallel shard.

The library (``libhsap.so``, C ABI in ``include/hsap.h``) holds the host
planner and the gfx950 HIP kernels; this package is its Python binding.  It
never falls back to a CPU path: without the built library every entry point
raises.
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    MAJOR_K,
    MAJOR_Q,
    MAJOR_Q_ALL,
    TILE_FULL,
    TILE_MASKED,
    AttnDesc,
    Executor,
    HsapError,
    ShardDesc,
    attn_bwd_bf16,
    attn_bwd_preprocess,
    attn_desc,
    attn_fwd_fused,
    convert_f32_bf16,
    doc_start,
    lib,
    lse_merge,
    partial_attn_bwd,
    partial_attn_bwd_runs,
    partial_attn_fwd,
    partial_attn_fwd_runs,
    plan,
    plan_runs,
    shard_desc,
    shard_gather,
)
