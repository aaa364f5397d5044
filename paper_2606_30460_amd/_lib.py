"""ctypes binding of libhsap (the C ABI declared in include/hsap.h).

Argument marshalling only: every function here checks shapes and dtypes,
passes raw pointers and sizes to the library and raises ``HsapError`` on a
non-OK status.  Device buffers are torch tensors (torch supplies memory and
the current HIP stream); host arrays are numpy arrays.  There is no fallback:
if the library is not built, or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "libhsap.so")

HSAP_OK = 0
HSAP_ERR_INVALID_ARG = 1
HSAP_ERR_CAPACITY = 2
HSAP_ERR_UNSUPPORTED = 3
HSAP_ERR_HIP = 4

LAYOUT_CONTIGUOUS = 0
LAYOUT_ZIGZAG = 1
TILE_FULL = 0
TILE_MASKED = 1
MAJOR_Q = 0
MAJOR_K = 1
MAJOR_Q_ALL = 2
MAX_MERGE_PARTS = 64

# Every symbol include/hsap.h declares.
EXPORTED = (
    "hsap_status_string", "hsap_last_error", "hsap_plan", "hsap_plan_runs", "hsap_split_length",
    "hsap_fwd_resident_workgroups", "hsap_load_matrix",
    "hsap_balance", "hsap_emit_forward", "hsap_emit_backward", "hsap_doc_start",
    "hsap_shard_gather", "hsap_partial_attn_fwd", "hsap_partial_attn_bwd", "hsap_partial_attn_fwd_runs", "hsap_attn_fwd_fused", "hsap_quantize_fp8", "hsap_quantize_fp8_noalloc",
    "hsap_partial_attn_fwd_fp8", "hsap_lse_merge", "hsap_attn_bwd_preprocess",
    "hsap_partial_attn_bwd_runs", "hsap_attn_bwd_bf16", "hsap_sum_parts", "hsap_convert_f32_bf16", "hsap_executor_create", "hsap_executor_destroy",
    "hsap_executor_plan", "hsap_executor_info", "hsap_executor_forward", "hsap_executor_partial_forward",
    "hsap_executor_merge", "hsap_executor_backward",
)

EXEC_BACKWARD = 1
EXEC_FUSED = 2


class HsapError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (_status_name(status), message))
        self.status = status


class ShardDesc(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int64), ("sp_degree", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("shard_id", ctypes.c_int32), ("block_m", ctypes.c_int32), ("block_n", ctypes.c_int32),
                ("batch", ctypes.c_int32)]

    @property
    def sequences(self) -> int:
        return max(int(self.batch), 1)

    @property
    def rows(self) -> int:
        """Local rows of one shard over the batch (B * N / P)."""
        return self.sequences * (self.total_tokens // self.sp_degree)

    @property
    def positions(self) -> int:
        """Positions over the batch (B * N)."""
        return self.sequences * self.total_tokens


class AttnDesc(ctypes.Structure):
    _fields_ = [("shard", ShardDesc), ("chunk_id", ctypes.c_int32), ("heads_q", ctypes.c_int32),
                ("heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float)]


class ExecInfo(ctypes.Structure):
    _fields_ = [("num_tiles", ctypes.c_int64), ("num_full_tiles", ctypes.c_int64), ("useful_pairs", ctypes.c_int64),
                ("num_runs_q", ctypes.c_int64), ("num_runs_k", ctypes.c_int64), ("num_runs_all", ctypes.c_int64),
                ("num_parts", ctypes.c_int32), ("split_length", ctypes.c_int32),
                ("chunks_with_tiles", ctypes.c_int32), ("final_q_tiles", ctypes.c_int32), ("chunk_mask", ctypes.c_uint64)]


_lib: Optional[ctypes.CDLL] = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SIG = {
    "hsap_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "hsap_last_error": (ctypes.c_char_p, []),
    "hsap_plan": (ctypes.c_int, [_P, _I32, _P, _P, _I64, _P, _P, _P]),
    "hsap_plan_runs": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _P, _P, _I64, _P, _P]),
    "hsap_split_length": (ctypes.c_int32, [_P, _I64, _I32, _I32]),
    "hsap_fwd_resident_workgroups": (ctypes.c_int, [_P, _P]),
    "hsap_load_matrix": (ctypes.c_int, [_P, _I32, _P, _P, _P]),
    "hsap_balance": (ctypes.c_int, [_I32, _P, _P, _P]),
    "hsap_emit_forward": (ctypes.c_int, [_I32, _P, _P, _P, _I64, _P, _P]),
    "hsap_emit_backward": (ctypes.c_int, [_I32, _P, _P, _P, _I64, _P, _P]),
    "hsap_doc_start": (ctypes.c_int, [_P, _I32, _I64, _P, _P]),
    "hsap_shard_gather": (ctypes.c_int, [_P, _P, _P, _I64, _P]),
    "hsap_partial_attn_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _I64, _P, _P, _P]),
    "hsap_partial_attn_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _P, _P]),
    "hsap_partial_attn_fwd_runs": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _I32, _P]),
    "hsap_attn_fwd_fused": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _P]),
    "hsap_quantize_fp8": (ctypes.c_int, [_P, _I32, _I64, _I32, _I32, _P, _P, _P, _P]),
    "hsap_quantize_fp8_noalloc": (ctypes.c_int, [_P, _I32, _I64, _I32, _I32, _P, _P, _P]),
    "hsap_partial_attn_fwd_fp8": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _I32, _P]),
    "hsap_lse_merge": (ctypes.c_int, [_I32, _P, _P, _I64, _I32, _I32, _P, _P, _P]),
    "hsap_attn_bwd_preprocess": (ctypes.c_int, [_P, _P, _I64, _I32, _I32, _P, _P]),
    "hsap_partial_attn_bwd_runs": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _I64, _P, _P, _P,
                                             _P]),
    "hsap_attn_bwd_bf16": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _I64, _P, _P, _P, _P]),
    "hsap_convert_f32_bf16": (ctypes.c_int, [_P, _P, _I64, _P]),
    "hsap_sum_parts": (ctypes.c_int, [_I32, _P, _I64, _P, _I32, _P]),
    "hsap_executor_create": (ctypes.c_int, [_P, _I32, _I32, _P]),
    "hsap_executor_destroy": (None, [_P]),
    "hsap_executor_plan": (ctypes.c_int, [_P, _P, _I32, _P]),
    "hsap_executor_info": (ctypes.c_int, [_P, _P]),
    "hsap_executor_forward": (ctypes.c_int, [_P, _P, _P, _P, _I32, _P, _P, _P]),
    "hsap_executor_partial_forward": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "hsap_executor_merge": (ctypes.c_int, [_P, _P, _P, _P]),
    "hsap_executor_backward": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libhsap.so is not built (%s); run __graft_entry__.build() or "
                               "python -m paper_2606_30460_amd.build" % LIB_PATH)
        # torch ships its own HIP runtime; loading torch first makes this library bind to that
        # one (loading ours first would leave torch with a runtime that sees no GPU)
        try:
            import torch  # noqa: F401
        except ImportError:  # pragma: no cover - host-only use of the planner
            pass
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _status_name(status: int) -> str:
    try:
        return lib().hsap_status_string(status).decode()
    except Exception:  # pragma: no cover
        return "status %d" % status


def _check(status: int) -> None:
    if status != HSAP_OK:
        raise HsapError(status, lib().hsap_last_error().decode())


def layout_code(layout) -> int:
    if isinstance(layout, str):
        return {"contiguous": LAYOUT_CONTIGUOUS, "zigzag": LAYOUT_ZIGZAG}[layout]
    return int(layout)


def shard_desc(total_tokens: int, sp_degree: int, layout, shard_id: int, block_m: int, block_n: int,
               batch: int = 1) -> ShardDesc:
    """Shard descriptor; ``total_tokens`` is one packed sequence's length, ``batch`` the number of
    such sequences per call (concatenated)."""
    return ShardDesc(int(total_tokens), int(sp_degree), layout_code(layout), int(shard_id), int(block_m), int(block_n),
                     int(batch))


def attn_desc(shard: ShardDesc, heads_q: int, heads_kv: int, head_dim: int, softmax_scale: float,
              chunk_id: int = 0) -> AttnDesc:
    return AttnDesc(shard=shard, chunk_id=int(chunk_id), heads_q=int(heads_q), heads_kv=int(heads_kv),
                    head_dim=int(head_dim), softmax_scale=float(softmax_scale))


def _ptr(a) -> int:
    """Raw address of a numpy array or torch tensor (None -> NULL)."""
    if a is None:
        return 0
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return int(a.data_ptr())


def _stream(stream) -> int:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _dev(t, dtype_name: str, what: str, numel: Optional[int] = None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("%s must be a device tensor" % what)
    if str(t.dtype) != "torch." + dtype_name:
        raise TypeError("%s must be %s, got %s" % (what, dtype_name, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if numel is not None and t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (what, t.numel(), numel))
    return t


# ---------------------------------------------------------------------------
# host planner
# ---------------------------------------------------------------------------

def plan(cu_seqlens, shard: ShardDesc) -> Dict[str, np.ndarray]:
    """hsap_plan with the two-call pattern.  Returns tiles int32 [T, 4],
    step_offsets int64 [P+1], useful_pairs int64 [P]."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    P = shard.sp_degree
    num = ctypes.c_int64(0)
    offs = np.zeros(max(P, 0) + 1, dtype=np.int64)
    pairs = np.zeros(max(P, 1), dtype=np.int64)
    st = lib().hsap_plan(_ptr(cu), len(cu) - 1, ctypes.byref(shard), None, 0, ctypes.byref(num),
                         _ptr(offs), _ptr(pairs))
    if st != HSAP_ERR_CAPACITY:
        _check(st)
    tiles = np.zeros((max(num.value, 1), 4), dtype=np.int32)
    _check(lib().hsap_plan(_ptr(cu), len(cu) - 1, ctypes.byref(shard), _ptr(tiles), tiles.shape[0],
                           ctypes.byref(num), _ptr(offs), _ptr(pairs)))
    return {"tiles": tiles[: num.value], "step_offsets": offs, "useful_pairs": pairs[:P]}


def plan_runs(shard: ShardDesc, tiles: np.ndarray, major: int, max_run_tiles: int = 0):
    """hsap_plan_runs.  Returns (sorted_tiles int32 [T, 4], runs int32 [R, 4] of (slot, tile, first, count),
    num_slots)."""
    tiles = np.ascontiguousarray(tiles, dtype=np.int32).reshape(-1, 4)
    sorted_tiles = np.zeros((max(len(tiles), 1), 4), dtype=np.int32)
    num = ctypes.c_int64(0)
    slots = ctypes.c_int32(0)
    st = lib().hsap_plan_runs(ctypes.byref(shard), _ptr(tiles), len(tiles), int(major), int(max_run_tiles),
                              _ptr(sorted_tiles), None, 0, ctypes.byref(num), ctypes.byref(slots))
    if st != HSAP_ERR_CAPACITY:
        _check(st)
    runs = np.zeros((max(num.value, 1), 4), dtype=np.int32)
    _check(lib().hsap_plan_runs(ctypes.byref(shard), _ptr(tiles), len(tiles), int(major), int(max_run_tiles),
                                _ptr(sorted_tiles), _ptr(runs), runs.shape[0], ctypes.byref(num),
                                ctypes.byref(slots)))
    return sorted_tiles[: len(tiles)], runs[: num.value], slots.value


def split_length(shard: ShardDesc, num_tiles: int, heads_q: int, resident_workgroups: int) -> int:
    """hsap_split_length: max_run_tiles for hsap_plan_runs (0 = no split)."""
    v = lib().hsap_split_length(ctypes.byref(shard), int(num_tiles), int(heads_q), int(resident_workgroups))
    if v < 0:
        raise HsapError(HSAP_ERR_INVALID_ARG, lib().hsap_last_error().decode())
    return v


def fwd_resident_workgroups(desc: AttnDesc) -> int:
    """hsap_fwd_resident_workgroups: partial-forward workgroups resident on the current device."""
    out = ctypes.c_int32(0)
    _check(lib().hsap_fwd_resident_workgroups(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def plan_into(cu_seqlens: np.ndarray, shard: ShardDesc, tiles_out: np.ndarray, step_offsets_out: np.ndarray,
              useful_pairs_out: np.ndarray) -> int:
    """hsap_plan into caller-provided host buffers (e.g. views of pinned memory).

    ``tiles_out`` int32 [capacity, 4]; returns the tile count."""
    num = ctypes.c_int64(0)
    _check(lib().hsap_plan(_ptr(cu_seqlens), len(cu_seqlens) - 1, ctypes.byref(shard), _ptr(tiles_out),
                           tiles_out.shape[0], ctypes.byref(num), _ptr(step_offsets_out), _ptr(useful_pairs_out)))
    return num.value


def load_matrix(cu_seqlens, shard: ShardDesc):
    """hsap_load_matrix: (tiles, pairs), int64 [P, P] indexed [shard r, chunk c]."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    P = shard.sp_degree
    tiles = np.zeros((P, P), dtype=np.int64)
    pairs = np.zeros((P, P), dtype=np.int64)
    _check(lib().hsap_load_matrix(_ptr(cu), len(cu) - 1, ctypes.byref(shard), _ptr(tiles), _ptr(pairs)))
    return tiles, pairs


def balance(cost):
    """hsap_balance: (exec_rank int32 [P, P], load int64 [P]) for block costs [P, P]."""
    cost = np.ascontiguousarray(cost, dtype=np.int64)
    if cost.ndim != 2 or cost.shape[0] != cost.shape[1]:
        raise ValueError("cost must be a square [P, P] matrix")
    P = cost.shape[0]
    exec_rank = np.zeros((P, P), dtype=np.int32)
    load = np.zeros(P, dtype=np.int64)
    _check(lib().hsap_balance(int(P), _ptr(cost), _ptr(exec_rank), _ptr(load)))
    return exec_rank, load


OP_SEND, OP_RECV, OP_COMPUTE, OP_MERGE = 0, 1, 2, 3
T_NONE, T_Q, T_KV, T_O, T_DQ, T_DKV, T_DO = -1, 0, 1, 2, 3, 4, 5


def _emit(fn, block_tiles, exec_rank):
    tiles = np.ascontiguousarray(block_tiles, dtype=np.int64)
    ex = np.ascontiguousarray(exec_rank, dtype=np.int32)
    P = tiles.shape[0]
    offs = np.zeros(P + 1, dtype=np.int64)
    stages = ctypes.c_int32(0)
    st = fn(int(P), _ptr(tiles), _ptr(ex), None, 0, _ptr(offs), ctypes.byref(stages))
    if st != HSAP_ERR_CAPACITY:
        _check(st)
    ops = np.zeros((max(int(offs[P]), 1), 8), dtype=np.int32)
    _check(fn(int(P), _ptr(tiles), _ptr(ex), _ptr(ops), int(offs[P]), _ptr(offs), ctypes.byref(stages)))
    return [ops[offs[e]:offs[e + 1]] for e in range(P)], int(stages.value)


def emit_forward(block_tiles, exec_rank):
    """hsap_emit_forward with the two-call pattern: (list of int32 [ops_e, 8] arrays per rank --
    fields op, tensor, peer, stage, shard, chunk, in_slot, out_slot -- and the number of stages)."""
    return _emit(lib().hsap_emit_forward, block_tiles, exec_rank)


def emit_backward(block_tiles, exec_rank):
    """hsap_emit_backward with the two-call pattern, as emit_forward."""
    return _emit(lib().hsap_emit_backward, block_tiles, exec_rank)


def plan_runs_into(shard: ShardDesc, tiles: np.ndarray, num_tiles: int, major: int, max_run_tiles: int,
                   sorted_out: np.ndarray, runs_out: np.ndarray):
    """hsap_plan_runs into caller-provided host buffers; returns (run count, slot count)."""
    num = ctypes.c_int64(0)
    slots = ctypes.c_int32(0)
    _check(lib().hsap_plan_runs(ctypes.byref(shard), _ptr(tiles), int(num_tiles), int(major), int(max_run_tiles),
                                _ptr(sorted_out), _ptr(runs_out), runs_out.shape[0], ctypes.byref(num),
                                ctypes.byref(slots)))
    return num.value, slots.value


# ---------------------------------------------------------------------------
# device entry points
# ---------------------------------------------------------------------------

def doc_start(cu_seqlens_dev, total_tokens: int, out, stream=None) -> None:
    _dev(cu_seqlens_dev, "int32", "cu_seqlens")
    _dev(out, "int32", "doc_start", total_tokens)
    _check(lib().hsap_doc_start(_ptr(cu_seqlens_dev), cu_seqlens_dev.numel() - 1, int(total_tokens), _ptr(out),
                                _stream(stream)))


def shard_gather(shard: ShardDesc, src, dst, stream=None) -> None:
    import torch
    if src.shape != dst.shape or src.dtype != dst.dtype or not (src.is_cuda and dst.is_cuda):
        raise ValueError("src and dst must be device tensors of one shape and dtype")
    if not (src.is_contiguous() and dst.is_contiguous()) or src.shape[0] != shard.positions:
        raise ValueError("src and dst must be contiguous with total_tokens x batch rows")
    row_bytes = src[0].numel() * src.element_size() if src.shape[0] else 0
    del torch
    _check(lib().hsap_shard_gather(ctypes.byref(shard), _ptr(src), _ptr(dst), int(row_bytes), _stream(stream)))


def _kv_base(t, chunk: int, n: int, hkv: int, d: int, elem: int, what: str) -> int:
    """Address of chunk 0 for k / v / dk / dv given either every chunk [P, n, Hkv, d] or chunk c alone."""
    if t.numel() == n * hkv * d:
        return _ptr(t) - int(chunk) * n * hkv * d * elem
    return _ptr(t)


def partial_attn_fwd(desc: AttnDesc, q, k, v, doc_start_dev, tiles_dev, o_part, lse_part, stream=None) -> None:
    """hsap_partial_attn_fwd: shard r's queries against chunk desc.chunk_id over that chunk's tiles (int32
    [T, 4], hsap_plan's order) -> o_part fp32 [n, Hq, d], lse_part fp32 [Hq, n].  k / v are every chunk
    [P, n, Hkv, d] or chunk chunk_id alone [n, Hkv, d]."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q, "bfloat16", "q", n * hq * d)
    for t, name in ((k, "k"), (v, "v")):
        _dev(t, "bfloat16", name)
        if t.numel() not in (n * hkv * d, P * n * hkv * d):
            raise ValueError("%s must hold one chunk or every chunk" % name)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    _dev(tiles_dev, "int32", "tiles")
    _dev(o_part, "float32", "o_part", n * hq * d)
    _dev(lse_part, "float32", "lse_part", hq * n)
    c = desc.chunk_id
    _check(lib().hsap_partial_attn_fwd(ctypes.byref(desc), _ptr(q), _kv_base(k, c, n, hkv, d, 2, "k"),
                                       _kv_base(v, c, n, hkv, d, 2, "v"), _ptr(doc_start_dev), _ptr(tiles_dev),
                                       tiles_dev.numel() // 4, _ptr(o_part), _ptr(lse_part), _stream(stream)))


def partial_attn_bwd(desc: AttnDesc, q, k, v, d_o, lse, delta, doc_start_dev, tiles_dev, dq_acc, dk_acc, dv_acc,
                     stream=None) -> None:
    """hsap_partial_attn_bwd: the gradients of partial_attn_fwd's partial (chunk desc.chunk_id, its tiles),
    accumulated (+=) into dq_acc fp32 [n, Hq, d] and dk_acc / dv_acc fp32 (every chunk [P, n, Hkv, d] or
    chunk chunk_id alone [n, Hkv, d], like k / v)."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q, "bfloat16", "q", n * hq * d)
    _dev(d_o, "bfloat16", "d_o", n * hq * d)
    _dev(lse, "float32", "lse", hq * n)
    _dev(delta, "float32", "delta", hq * n)
    for t, name, dt in ((k, "k", "bfloat16"), (v, "v", "bfloat16"), (dk_acc, "dk_acc", "float32"),
                        (dv_acc, "dv_acc", "float32")):
        _dev(t, dt, name)
        if t.numel() not in (n * hkv * d, P * n * hkv * d):
            raise ValueError("%s must hold one chunk or every chunk" % name)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    _dev(tiles_dev, "int32", "tiles")
    _dev(dq_acc, "float32", "dq_acc", n * hq * d)
    c = desc.chunk_id
    _check(lib().hsap_partial_attn_bwd(ctypes.byref(desc), _ptr(q), _kv_base(k, c, n, hkv, d, 2, "k"),
                                       _kv_base(v, c, n, hkv, d, 2, "v"), _ptr(d_o), _ptr(lse), _ptr(delta),
                                       _ptr(doc_start_dev), _ptr(tiles_dev), tiles_dev.numel() // 4, _ptr(dq_acc),
                                       _kv_base(dk_acc, c, n, hkv, d, 4, "dk"), _kv_base(dv_acc, c, n, hkv, d, 4, "dv"),
                                       _stream(stream)))


def partial_attn_fwd_runs(desc: AttnDesc, q, k, v, doc_start_dev, tiles_dev, runs_dev, o_part, lse_part,
                     stream=None, kv_chunk: Optional[int] = None) -> None:
    """hsap_partial_attn_fwd_runs.  k / v are [P, n, Hkv, d] (every chunk, sharded order), or, with
    ``kv_chunk`` = c, [n, Hkv, d] holding chunk c alone (every run passed must be of chunk c):
    the library then gets the address chunk 0 would have, and reads only chunk c's rows."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q, "bfloat16", "q", n * hq * d)
    kv_rows = P if kv_chunk is None else 1
    _dev(k, "bfloat16", "k", kv_rows * n * hkv * d)
    _dev(v, "bfloat16", "v", kv_rows * n * hkv * d)
    kv_shift = 0
    if kv_chunk is not None:
        if not 0 <= int(kv_chunk) < P:
            raise ValueError("kv_chunk %d outside [0, %d)" % (kv_chunk, P))
        kv_shift = int(kv_chunk) * n * hkv * d * 2
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    _dev(tiles_dev, "int32", "tiles")
    _dev(runs_dev, "int32", "runs")
    _dev(o_part, "float32", "o_part")
    _dev(lse_part, "float32", "lse_part")
    slots = o_part.numel() // (n * hq * d)
    if o_part.numel() != slots * n * hq * d or lse_part.numel() != slots * hq * n or slots < 1:
        raise ValueError("o_part / lse_part must hold a whole number of [n, Hq, d] / [Hq, n] slots")
    _check(lib().hsap_partial_attn_fwd_runs(ctypes.byref(desc), _ptr(q), _ptr(k) - kv_shift, _ptr(v) - kv_shift,
                                       _ptr(doc_start_dev),
                                       _ptr(tiles_dev), _ptr(runs_dev), runs_dev.numel() // 4, _ptr(o_part),
                                       _ptr(lse_part), int(slots), _stream(stream)))


QUANT_SPLIT = 32


def quantize_fp8(x, codes, scale, workspace, stream=None) -> None:
    """hsap_quantize_fp8: x bf16 [G, rows, H, d] -> codes uint8 (same shape), scale fp32 [G, H];
    workspace fp32 [G * H * QUANT_SPLIT]."""
    if x.dim() != 4:
        raise ValueError("x must be [groups, rows, heads, head_dim]")
    G, rows, H, d = x.shape
    _dev(x, "bfloat16", "x")
    _dev(codes, "uint8", "codes", x.numel())
    _dev(scale, "float32", "scale", G * H)
    _dev(workspace, "float32", "workspace", G * H * QUANT_SPLIT)
    _check(lib().hsap_quantize_fp8(_ptr(x), int(G), int(rows), int(H), int(d), _ptr(codes), _ptr(scale),
                                   _ptr(workspace), _stream(stream)))


QUANT_NOALLOC_MAX_SLICES = 4096


def quantize_fp8_noalloc(x, codes, scale, stream=None) -> None:
    """hsap_quantize_fp8_noalloc: hsap_quantize_fp8 with the per-range maxima in the library's own
    fixed scratch array (no workspace; at most QUANT_NOALLOC_MAX_SLICES groups x heads)."""
    if x.dim() != 4:
        raise ValueError("x must be [groups, rows, heads, head_dim]")
    G, rows, H, d = x.shape
    _dev(x, "bfloat16", "x")
    _dev(codes, "uint8", "codes", x.numel())
    _dev(scale, "float32", "scale", G * H)
    _check(lib().hsap_quantize_fp8_noalloc(_ptr(x), int(G), int(rows), int(H), int(d), _ptr(codes), _ptr(scale),
                                           _stream(stream)))


def partial_attn_fwd_fp8(desc: AttnDesc, q8, k8, v, q_scale, k_scale, doc_start_dev, tiles_dev, runs_dev, o_part,
                         lse_part, stream=None) -> None:
    """hsap_partial_attn_fwd_fp8: the partial forward with e4m3 Q [n, Hq, d] and K [P, n, Hkv, d] and their
    scales [Hq] and [P, Hkv] (hsap_quantize_fp8); V, outputs and lists as for partial_attn_fwd_runs."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q8, "uint8", "q8", n * hq * d)
    _dev(k8, "uint8", "k8", P * n * hkv * d)
    _dev(v, "bfloat16", "v", P * n * hkv * d)
    _dev(q_scale, "float32", "q_scale", hq)
    _dev(k_scale, "float32", "k_scale", P * hkv)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    _dev(tiles_dev, "int32", "tiles")
    _dev(runs_dev, "int32", "runs")
    _dev(o_part, "float32", "o_part")
    _dev(lse_part, "float32", "lse_part")
    slots = o_part.numel() // (n * hq * d)
    if o_part.numel() != slots * n * hq * d or lse_part.numel() != slots * hq * n or slots < 1:
        raise ValueError("o_part / lse_part must hold a whole number of [n, Hq, d] / [Hq, n] slots")
    _check(lib().hsap_partial_attn_fwd_fp8(ctypes.byref(desc), _ptr(q8), _ptr(k8), _ptr(v), _ptr(q_scale),
                                           _ptr(k_scale), _ptr(doc_start_dev), _ptr(tiles_dev), _ptr(runs_dev),
                                           runs_dev.numel() // 4, _ptr(o_part), _ptr(lse_part), int(slots),
                                           _stream(stream)))


def attn_fwd_fused(desc: AttnDesc, q, k, v, doc_start_dev, tiles_dev, runs_dev, o_out, lse_out, stream=None) -> None:
    """hsap_attn_fwd_fused over MAJOR_Q_ALL runs: final bf16 O and LSE in one pass."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q, "bfloat16", "q", n * hq * d)
    _dev(k, "bfloat16", "k", P * n * hkv * d)
    _dev(v, "bfloat16", "v", P * n * hkv * d)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    _dev(tiles_dev, "int32", "tiles")
    _dev(runs_dev, "int32", "runs")
    _dev(o_out, "bfloat16", "o_out", n * hq * d)
    _dev(lse_out, "float32", "lse_out", hq * n)
    _check(lib().hsap_attn_fwd_fused(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(doc_start_dev),
                                     _ptr(tiles_dev), _ptr(runs_dev), runs_dev.numel() // 4, _ptr(o_out),
                                     _ptr(lse_out), _stream(stream)))


def lse_merge(o_parts: Sequence, lse_parts: Sequence, n: int, heads_q: int, head_dim: int, o_out, lse_out,
              stream=None) -> None:
    if len(o_parts) != len(lse_parts) or not o_parts:
        raise ValueError("need matching, non-empty part lists")
    for i, (o, l) in enumerate(zip(o_parts, lse_parts)):
        _dev(o, "float32", "o_parts[%d]" % i, n * heads_q * head_dim)
        _dev(l, "float32", "lse_parts[%d]" % i, heads_q * n)
    _dev(o_out, "bfloat16", "o_out", n * heads_q * head_dim)
    _dev(lse_out, "float32", "lse_out", heads_q * n)
    np_ = len(o_parts)
    o_arr = (ctypes.c_void_p * np_)(*[_ptr(t) for t in o_parts])
    l_arr = (ctypes.c_void_p * np_)(*[_ptr(t) for t in lse_parts])
    _check(lib().hsap_lse_merge(np_, o_arr, l_arr, int(n), int(heads_q), int(head_dim), _ptr(o_out), _ptr(lse_out),
                                _stream(stream)))


def attn_bwd_preprocess(o, d_o, n: int, heads_q: int, head_dim: int, delta, stream=None) -> None:
    _dev(o, "bfloat16", "o", n * heads_q * head_dim)
    _dev(d_o, "bfloat16", "d_o", n * heads_q * head_dim)
    _dev(delta, "float32", "delta", heads_q * n)
    _check(lib().hsap_attn_bwd_preprocess(_ptr(o), _ptr(d_o), int(n), int(heads_q), int(head_dim), _ptr(delta),
                                          _stream(stream)))


def partial_attn_bwd_runs(desc: AttnDesc, q, k, v, d_o, lse, delta, doc_start_dev, tiles_k_dev, runs_k_dev, tiles_q_dev,
                     runs_q_dev, dq_acc, dk_acc, dv_acc, stream=None, kv_chunk: Optional[int] = None) -> None:
    """hsap_partial_attn_bwd_runs.  Either run list may be None to skip its kernel.  With ``kv_chunk`` = c,
    k, v, dk_acc and dv_acc are [n, Hkv, d] tensors of chunk c alone (every run passed must be of
    chunk c), passed as the addresses chunk 0 would have."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    kv_rows = P if kv_chunk is None else 1
    kv_shift = 0
    if kv_chunk is not None:
        if not 0 <= int(kv_chunk) < P:
            raise ValueError("kv_chunk %d outside [0, %d)" % (kv_chunk, P))
        kv_shift = int(kv_chunk) * n * hkv * d
    _dev(q, "bfloat16", "q", n * hq * d)
    _dev(k, "bfloat16", "k", kv_rows * n * hkv * d)
    _dev(v, "bfloat16", "v", kv_rows * n * hkv * d)
    _dev(d_o, "bfloat16", "d_o", n * hq * d)
    _dev(lse, "float32", "lse", hq * n)
    _dev(delta, "float32", "delta", hq * n)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    for t, name in ((tiles_k_dev, "tiles_k"), (runs_k_dev, "runs_k"), (tiles_q_dev, "tiles_q"), (runs_q_dev, "runs_q")):
        if t is not None:
            _dev(t, "int32", name)
    _dev(dq_acc, "float32", "dq_acc", n * hq * d)
    _dev(dk_acc, "float32", "dk_acc", kv_rows * n * hkv * d)
    _dev(dv_acc, "float32", "dv_acc", kv_rows * n * hkv * d)
    nk = runs_k_dev.numel() // 4 if runs_k_dev is not None else 0
    nq = runs_q_dev.numel() // 4 if runs_q_dev is not None else 0
    _check(lib().hsap_partial_attn_bwd_runs(ctypes.byref(desc), _ptr(q), _ptr(k) - 2 * kv_shift, _ptr(v) - 2 * kv_shift,
                                       _ptr(d_o), _ptr(lse), _ptr(delta), _ptr(doc_start_dev), _ptr(tiles_k_dev),
                                       _ptr(runs_k_dev), nk, _ptr(tiles_q_dev), _ptr(runs_q_dev), nq, _ptr(dq_acc),
                                       _ptr(dk_acc) - 4 * kv_shift, _ptr(dv_acc) - 4 * kv_shift, _stream(stream)))


def sum_parts(parts, out, stream=None) -> None:
    """hsap_sum_parts: out = parts[0] + parts[1] + ... (fp32, in order), out fp32 or bf16 of the parts' size."""
    count = parts[0].numel()
    for i, p in enumerate(parts):
        _dev(p, "float32", "parts[%d]" % i, count)
    if str(out.dtype) not in ("torch.float32", "torch.bfloat16"):
        raise TypeError("out must be float32 or bfloat16")
    _dev(out, str(out.dtype)[6:], "out", count)
    arr = (ctypes.c_void_p * len(parts))(*[_ptr(p) for p in parts])
    _check(lib().hsap_sum_parts(len(parts), arr, count, _ptr(out), int(str(out.dtype) == "torch.bfloat16"),
                                _stream(stream)))


def attn_bwd_bf16(desc: AttnDesc, q, k, v, d_o, lse, delta, doc_start_dev, tiles_k_dev, runs_k_dev, tiles_all_dev,
                  runs_all_dev, dq, dk, dv, stream=None) -> None:
    """hsap_attn_bwd_bf16: final bf16 gradients over every chunk (MAJOR_K and MAJOR_Q_ALL lists)."""
    s = desc.shard
    n = s.rows
    hq, hkv, d, P = desc.heads_q, desc.heads_kv, desc.head_dim, s.sp_degree
    _dev(q, "bfloat16", "q", n * hq * d)
    _dev(k, "bfloat16", "k", P * n * hkv * d)
    _dev(v, "bfloat16", "v", P * n * hkv * d)
    _dev(d_o, "bfloat16", "d_o", n * hq * d)
    _dev(lse, "float32", "lse", hq * n)
    _dev(delta, "float32", "delta", hq * n)
    _dev(doc_start_dev, "int32", "doc_start", s.positions)
    for t, name in ((tiles_k_dev, "tiles_k"), (runs_k_dev, "runs_k"), (tiles_all_dev, "tiles_all"),
                    (runs_all_dev, "runs_all")):
        _dev(t, "int32", name)
    _dev(dq, "bfloat16", "dq", n * hq * d)
    _dev(dk, "bfloat16", "dk", P * n * hkv * d)
    _dev(dv, "bfloat16", "dv", P * n * hkv * d)
    _check(lib().hsap_attn_bwd_bf16(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(d_o), _ptr(lse), _ptr(delta),
                                    _ptr(doc_start_dev), _ptr(tiles_k_dev), _ptr(runs_k_dev), runs_k_dev.numel() // 4,
                                    _ptr(tiles_all_dev), _ptr(runs_all_dev), runs_all_dev.numel() // 4, _ptr(dq),
                                    _ptr(dk), _ptr(dv), _stream(stream)))


def convert_f32_bf16(src, dst, stream=None) -> None:
    _dev(src, "float32", "src")
    _dev(dst, "bfloat16", "dst", src.numel())
    _check(lib().hsap_convert_f32_bf16(_ptr(src), _ptr(dst), src.numel(), _stream(stream)))


# ---------------------------------------------------------------------------
# step executor
# ---------------------------------------------------------------------------

class Executor:
    """hsap_executor: plan a packed batch, then run the shard's forward and
    backward, one library call each.

    ``max_run_tiles``: -1 picks the q-major split per plan, 0 never splits.
    Tensors are checked once per call (dtype, size, contiguity); all calls
    should use the same stream.
    """

    def __init__(self, desc: AttnDesc, backward: bool = False, fused: bool = False, max_run_tiles: int = -1):
        self.desc = desc
        s = desc.shard
        self.n = s.rows
        self.P = s.sp_degree
        self._q_numel = self.n * desc.heads_q * desc.head_dim
        self._kv_numel = self.P * self.n * desc.heads_kv * desc.head_dim
        self._lse_numel = desc.heads_q * self.n
        opts = (EXEC_BACKWARD if backward else 0) | (EXEC_FUSED if fused else 0)
        handle = ctypes.c_void_p(0)
        _check(lib().hsap_executor_create(ctypes.byref(desc), opts, int(max_run_tiles), ctypes.byref(handle)))
        self._h = handle

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().hsap_executor_destroy(self._h)
        self._h = None

    def __del__(self):  # pragma: no cover - interpreter shutdown order
        try:
            self.close()
        except Exception:
            pass

    def _handle(self):
        if self._h is None:
            raise RuntimeError("executor is closed")
        return self._h

    def plan(self, cu_seqlens: np.ndarray, stream=None) -> None:
        """Plan one batch (host int32 cu_seqlens [num_docs + 1])."""
        cu = cu_seqlens
        if not (isinstance(cu, np.ndarray) and cu.dtype == np.int32 and cu.flags.c_contiguous):
            cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        _check(lib().hsap_executor_plan(self._handle(), cu.ctypes.data, len(cu) - 1, _stream(stream)))

    def info(self) -> Dict[str, int]:
        out = ExecInfo()
        _check(lib().hsap_executor_info(self._handle(), ctypes.byref(out)))
        return {name: int(getattr(out, name)) for name, _ in ExecInfo._fields_}

    def forward(self, q, k, v, o_out, lse_out, fused: bool = False, stream=None) -> None:
        _dev(q, "bfloat16", "q", self._q_numel)
        _dev(k, "bfloat16", "k", self._kv_numel)
        _dev(v, "bfloat16", "v", self._kv_numel)
        _dev(o_out, "bfloat16", "o_out", self._q_numel)
        _dev(lse_out, "float32", "lse_out", self._lse_numel)
        _check(lib().hsap_executor_forward(self._handle(), _ptr(q), _ptr(k), _ptr(v), int(bool(fused)), _ptr(o_out),
                                           _ptr(lse_out), _stream(stream)))

    def partial_forward(self, q, k, v, o_out, lse_out, stream=None) -> None:
        """First stage of forward(fused=False): partial attention into the executor's partials (q-tiles
        with a single part straight into o_out / lse_out)."""
        _dev(q, "bfloat16", "q", self._q_numel)
        _dev(k, "bfloat16", "k", self._kv_numel)
        _dev(v, "bfloat16", "v", self._kv_numel)
        _dev(o_out, "bfloat16", "o_out", self._q_numel)
        _dev(lse_out, "float32", "lse_out", self._lse_numel)
        _check(lib().hsap_executor_partial_forward(self._handle(), _ptr(q), _ptr(k), _ptr(v), _ptr(o_out),
                                                   _ptr(lse_out), _stream(stream)))

    def merge(self, o_out, lse_out, stream=None) -> None:
        """Second stage: LSE merge of the partials into o_out / lse_out (the rows the first stage left)."""
        _dev(o_out, "bfloat16", "o_out", self._q_numel)
        _dev(lse_out, "float32", "lse_out", self._lse_numel)
        _check(lib().hsap_executor_merge(self._handle(), _ptr(o_out), _ptr(lse_out), _stream(stream)))

    def backward(self, q, k, v, d_o, o, lse, dq, dk, dv, stream=None) -> None:
        _dev(q, "bfloat16", "q", self._q_numel)
        _dev(k, "bfloat16", "k", self._kv_numel)
        _dev(v, "bfloat16", "v", self._kv_numel)
        _dev(d_o, "bfloat16", "d_o", self._q_numel)
        _dev(o, "bfloat16", "o", self._q_numel)
        _dev(lse, "float32", "lse", self._lse_numel)
        _dev(dq, "bfloat16", "dq", self._q_numel)
        _dev(dk, "bfloat16", "dk", self._kv_numel)
        _dev(dv, "bfloat16", "dv", self._kv_numel)
        _check(lib().hsap_executor_backward(self._handle(), _ptr(q), _ptr(k), _ptr(v), _ptr(d_o), _ptr(o), _ptr(lse),
                                            _ptr(dq), _ptr(dk), _ptr(dv), _stream(stream)))
