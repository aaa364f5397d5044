"""The C ABI without a GPU: the library loads, exports what include/hsap.h declares,
and rejects malformed arguments before launching anything."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_30460_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "hsap.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hsap_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_what_binding_lists():
    assert _declared() == sorted(L.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = L.lib()
    for name in _declared():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_status_strings():
    lib = L.lib()
    for code, name in [(0, "HSAP_OK"), (1, "HSAP_ERR_INVALID_ARG"), (2, "HSAP_ERR_CAPACITY"),
                       (3, "HSAP_ERR_UNSUPPORTED"), (4, "HSAP_ERR_HIP")]:
        assert lib.hsap_status_string(code).decode() == name


def test_struct_layouts():
    assert ctypes.sizeof(L.ShardDesc) == 32
    assert ctypes.sizeof(L.AttnDesc) == 56
    assert L.AttnDesc.chunk_id.offset == 32 and L.AttnDesc.heads_q.offset == 36


def _status(fn, *args):
    return fn(*args)


def test_plan_rejects_bad_cu_seqlens():
    lib = L.lib()
    d = L.shard_desc(64, 2, "contiguous", 0, 16, 16)
    num = ctypes.c_int64(-1)
    for cu in ([1, 64], [0, 30, 20, 64], [0, 63], [0, 65]):
        arr = np.asarray(cu, dtype=np.int32)
        st = lib.hsap_plan(arr.ctypes.data, len(arr) - 1, ctypes.byref(d), None, 0, ctypes.byref(num), None, None)
        assert st == L.HSAP_ERR_INVALID_ARG, cu
        assert lib.hsap_last_error().decode()


@pytest.mark.parametrize("bad", [
    dict(total_tokens=63, sp_degree=2),                 # N % P
    dict(total_tokens=64, sp_degree=4, layout=1),       # zigzag needs N % 2P ... 64 % 8 == 0 but BM must divide 8
    dict(shard_id=2),                                   # shard out of range
    dict(block_m=24),                                   # BM does not divide n
    dict(block_n=0),
    dict(layout=7),
    dict(sp_degree=0),
])
def test_plan_rejects_bad_shard(bad):
    lib = L.lib()
    args = dict(total_tokens=64, sp_degree=2, layout=0, shard_id=0, block_m=16, block_n=16)
    args.update(bad)
    d = L.ShardDesc(args["total_tokens"], args["sp_degree"], args["layout"], args["shard_id"], args["block_m"],
                    args["block_n"])
    cu = np.asarray([0, args["total_tokens"]], dtype=np.int32)
    num = ctypes.c_int64(-1)
    st = lib.hsap_plan(cu.ctypes.data, 1, ctypes.byref(d), None, 0, ctypes.byref(num), None, None)
    assert st == L.HSAP_ERR_INVALID_ARG


def test_plan_two_call_capacity():
    lib = L.lib()
    d = L.shard_desc(256, 2, "zigzag", 1, 32, 32)
    cu = np.asarray([0, 5, 100, 256], dtype=np.int32)
    num = ctypes.c_int64(0)
    offs = np.zeros(3, dtype=np.int64)
    st = lib.hsap_plan(cu.ctypes.data, 3, ctypes.byref(d), None, 0, ctypes.byref(num), offs.ctypes.data, None)
    assert st == L.HSAP_ERR_CAPACITY and num.value > 0 and offs[-1] == num.value
    small = np.zeros((num.value - 1, 4), dtype=np.int32)
    st = lib.hsap_plan(cu.ctypes.data, 3, ctypes.byref(d), small.ctypes.data, len(small), ctypes.byref(num), None,
                       None)
    assert st == L.HSAP_ERR_CAPACITY
    full = np.zeros((num.value, 4), dtype=np.int32)
    st = lib.hsap_plan(cu.ctypes.data, 3, ctypes.byref(d), full.ctypes.data, len(full), ctypes.byref(num), None, None)
    assert st == L.HSAP_OK


def test_plan_runs_rejects_non_canonical_list():
    d = L.shard_desc(256, 2, "contiguous", 1, 32, 32)
    p = L.plan([0, 256], d)
    tiles = p["tiles"].copy()
    tiles[[0, 1]] = tiles[[1, 0]]
    with pytest.raises(L.HsapError) as e:
        L.plan_runs(d, tiles, L.MAJOR_Q, 0)
    assert e.value.status == L.HSAP_ERR_INVALID_ARG


def _attn_desc(**over):
    s = dict(total_tokens=1024, sp_degree=2, layout=0, shard_id=0, block_m=128, block_n=128)
    s.update({k: v for k, v in over.items() if k in s})
    a = dict(heads_q=4, heads_kv=2, head_dim=128, softmax_scale=0.088)
    a.update({k: v for k, v in over.items() if k in a})
    return L.AttnDesc(L.ShardDesc(**s), **a)


@pytest.mark.parametrize("over,code", [
    (dict(head_dim=96), L.HSAP_ERR_UNSUPPORTED),
    (dict(heads_q=3), L.HSAP_ERR_INVALID_ARG),
    (dict(softmax_scale=0.0), L.HSAP_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), L.HSAP_ERR_INVALID_ARG),
    (dict(block_m=96, total_tokens=768 * 2), L.HSAP_ERR_UNSUPPORTED),
    (dict(block_n=32), L.HSAP_ERR_UNSUPPORTED),
])
def test_forward_validates_before_launch(over, code):
    lib = L.lib()
    d = _attn_desc(**over)
    fake = ctypes.c_void_p(4096)     # never dereferenced: validation fails first
    st = lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, 1, fake, fake, 1, None)
    assert st == code, lib.hsap_last_error().decode()


def test_tile_list_entry_points_validate_before_launch():
    # the boundary's tile-list forms: chunk_id, the list length and the outputs are checked first
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    for over, code in [(dict(chunk_id=2), L.HSAP_ERR_INVALID_ARG), (dict(chunk_id=-1), L.HSAP_ERR_INVALID_ARG),
                       (dict(head_dim=96), L.HSAP_ERR_UNSUPPORTED), (dict(block_n=32), L.HSAP_ERR_UNSUPPORTED)]:
        d = _attn_desc(**over)
        d.chunk_id = over.get("chunk_id", 1)
        st = lib.hsap_partial_attn_fwd(ctypes.byref(d), fake, fake, fake, fake, fake, 3, fake, fake, None)
        assert st == code, (over, lib.hsap_last_error().decode())
        st = lib.hsap_partial_attn_bwd(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, 3, fake, fake,
                                       fake, None)
        assert st == code, (over, lib.hsap_last_error().decode())
    d = _attn_desc()
    d.chunk_id = 1
    assert lib.hsap_partial_attn_fwd(ctypes.byref(d), fake, fake, fake, fake, fake, -1, fake, fake, None) == \
        L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_partial_attn_fwd(ctypes.byref(d), fake, fake, fake, fake, None, 3, fake, fake, None) == \
        L.HSAP_ERR_INVALID_ARG                                   # no list
    assert lib.hsap_partial_attn_fwd(ctypes.byref(d), fake, fake, fake, fake, fake, 3, None, fake, None) == \
        L.HSAP_ERR_INVALID_ARG                                   # no output
    assert lib.hsap_partial_attn_bwd(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, 0, fake, fake,
                                     fake, None) == L.HSAP_OK    # an empty list adds nothing
    # the dK/dV kernel gathers at most 2048 q-tiles per k-tile in LDS
    big = _attn_desc(total_tokens=2 * 2049 * 64, block_m=64, block_n=64)
    big.chunk_id = 0
    st = lib.hsap_partial_attn_bwd(ctypes.byref(big), fake, fake, fake, fake, fake, fake, fake, fake, 3, fake, fake,
                                   fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED and "2048" in lib.hsap_last_error().decode()


def test_forward_rejects_256_row_tiles_beyond_packed_descriptors():
    # the direct-to-LDS kernel (the only 256-row one) packs a tile's chunk into 8 bits: more than
    # 256 chunks are rejected before any launch (128-row tiles fall back to the register-staged
    # kernel instead)
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    d = _attn_desc(block_m=256, block_n=128, sp_degree=257, total_tokens=257 * 256)
    st = lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, 1, fake, fake, 1, None)
    assert st == L.HSAP_ERR_UNSUPPORTED, lib.hsap_last_error().decode()
    assert "256" in lib.hsap_last_error().decode()


def test_forward_rejects_null_and_misaligned():
    lib = L.lib()
    d = _attn_desc()
    fake = ctypes.c_void_p(4096)
    st = lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), None, fake, fake, fake, fake, fake, 1, fake, fake, 1, None)
    assert st == L.HSAP_ERR_INVALID_ARG
    odd = ctypes.c_void_p(4098)
    st = lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), odd, fake, fake, fake, fake, fake, 1, fake, fake, 1, None)
    assert st == L.HSAP_ERR_INVALID_ARG
    st = lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, 1, fake, fake, 0, None)
    assert st == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_partial_attn_fwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, 0, fake, fake, 1, None) == 0


def test_fused_forward_validates_before_launch():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    st = lib.hsap_attn_fwd_fused(ctypes.byref(_attn_desc(head_dim=96)), fake, fake, fake, fake, fake, fake, 1, fake,
                                 fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED
    st = lib.hsap_attn_fwd_fused(ctypes.byref(_attn_desc()), fake, fake, fake, fake, fake, fake, 1, None, fake, None)
    assert st == L.HSAP_ERR_INVALID_ARG


def test_fp8_entry_points_validate_before_launch():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    st = lib.hsap_partial_attn_fwd_fp8(ctypes.byref(_attn_desc(head_dim=64)), fake, fake, fake, fake, fake, fake, fake,
                                       fake, 1, fake, fake, 1, None)
    assert st == L.HSAP_ERR_UNSUPPORTED                      # fp8 scores need head_dim 128
    st = lib.hsap_partial_attn_fwd_fp8(ctypes.byref(_attn_desc()), fake, fake, fake, None, fake, fake, fake, fake, 1,
                                       fake, fake, 1, None)
    assert st == L.HSAP_ERR_INVALID_ARG                      # no q_scale
    st = lib.hsap_partial_attn_fwd_fp8(ctypes.byref(_attn_desc()), ctypes.c_void_p(4104), fake, fake, fake, fake,
                                       fake, fake, fake, 1, fake, fake, 1, None)
    assert st == L.HSAP_ERR_INVALID_ARG                      # q8 not 16-byte aligned
    assert lib.hsap_quantize_fp8(fake, 1, 4, 2, 12, fake, fake, fake, None) == L.HSAP_ERR_INVALID_ARG   # d % 8
    assert lib.hsap_quantize_fp8(fake, 0, 4, 2, 16, fake, fake, fake, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_quantize_fp8(ctypes.c_void_p(4100), 1, 4, 2, 16, fake, fake, fake, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_quantize_fp8(fake, 1, 4, 2, 16, None, fake, fake, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_quantize_fp8(fake, 1, 4, 2, 16, fake, fake, None, None) == L.HSAP_ERR_INVALID_ARG


def test_backward_validates_before_launch():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    d = _attn_desc(block_m=32, total_tokens=64 * 2, block_n=32)
    st = lib.hsap_partial_attn_bwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 1, fake,
                                   fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED
    d = _attn_desc(head_dim=64, block_n=128)
    st = lib.hsap_partial_attn_bwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 1, fake,
                                   fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED
    d = _attn_desc()
    st = lib.hsap_partial_attn_bwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, None, None, 1, fake,
                                   fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_INVALID_ARG


def test_backward_rejects_dq_beyond_packed_descriptors():
    # the dQ kernel packs a tile's chunk into 8 bits: more than 256 chunks are rejected before any
    # launch when q-major runs are passed (the dK/dV kernel alone has no such limit)
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    d = _attn_desc(sp_degree=260, total_tokens=260 * 128)
    for fn in (lib.hsap_partial_attn_bwd_runs, lib.hsap_attn_bwd_bf16):
        st = fn(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 0, fake, fake, 1, fake, fake,
                fake, None)
        assert st == L.HSAP_ERR_UNSUPPORTED, lib.hsap_last_error().decode()
        assert "256" in lib.hsap_last_error().decode()


def test_backward_shapes_of_256_row_tiles():
    # 256-row q-tiles have a backward for head_dim 128 only; a rejected shape launches nothing
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    d = _attn_desc(block_m=256, head_dim=64, block_n=64, total_tokens=2048)
    st = lib.hsap_partial_attn_bwd_runs(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 1, fake,
                                   fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED


def test_bf16_backward_validates_before_launch():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    d = _attn_desc(block_m=32, total_tokens=64 * 2, block_n=32)
    st = lib.hsap_attn_bwd_bf16(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 1, fake,
                                fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_UNSUPPORTED
    d = _attn_desc()
    st = lib.hsap_attn_bwd_bf16(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, None, None, 1, fake,
                                fake, 1, fake, fake, fake, None)
    assert st == L.HSAP_ERR_INVALID_ARG
    st = lib.hsap_attn_bwd_bf16(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 1, fake,
                                fake, 1, ctypes.c_void_p(4098), fake, fake, None)
    assert st == L.HSAP_ERR_INVALID_ARG                          # dq not 8-byte aligned
    assert lib.hsap_attn_bwd_bf16(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, fake, 0, fake,
                                  fake, 0, fake, fake, fake, None) == L.HSAP_OK   # nothing to do


def test_merge_and_helpers_validate():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)
    arr = (ctypes.c_void_p * 1)(4096)
    assert lib.hsap_lse_merge(0, arr, arr, 10, 2, 128, fake, fake, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_lse_merge(65, arr, arr, 10, 2, 128, fake, fake, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_lse_merge(1, arr, arr, 10, 2, 96, fake, fake, None) == L.HSAP_ERR_UNSUPPORTED
    assert lib.hsap_attn_bwd_preprocess(fake, fake, 10, 2, 80, fake, None) == L.HSAP_ERR_UNSUPPORTED
    assert lib.hsap_convert_f32_bf16(fake, fake, -1, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_convert_f32_bf16(None, None, 0, None) == L.HSAP_OK
    assert lib.hsap_doc_start(fake, 0, 10, fake, None) == L.HSAP_ERR_INVALID_ARG
    d = L.shard_desc(100, 3, "contiguous", 0, 1, 1)
    assert lib.hsap_shard_gather(ctypes.byref(d), fake, fake, 16, None) == L.HSAP_ERR_INVALID_ARG
    d = L.shard_desc(96, 3, "contiguous", 0, 1, 1)
    assert lib.hsap_shard_gather(ctypes.byref(d), fake, fake, 12, None) == L.HSAP_ERR_INVALID_ARG


def test_load_matrix_and_balance_validate():
    lib = L.lib()
    cu = np.asarray([0, 1024], dtype=np.int32)
    out = np.zeros(4, dtype=np.int64)
    s = L.shard_desc(1024, 2, "contiguous", 0, 128, 128)
    assert lib.hsap_load_matrix(cu.ctypes.data, 1, ctypes.byref(s), None, None) == L.HSAP_ERR_INVALID_ARG
    bad = np.asarray([0, 1000], dtype=np.int32)               # does not end at N
    assert lib.hsap_load_matrix(bad.ctypes.data, 1, ctypes.byref(s), out.ctypes.data, None) == L.HSAP_ERR_INVALID_ARG
    odd = L.shard_desc(1000, 2, "contiguous", 0, 128, 128)    # BM does not divide n
    assert lib.hsap_load_matrix(cu.ctypes.data, 1, ctypes.byref(odd), out.ctypes.data, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_load_matrix(cu.ctypes.data, 1, ctypes.byref(s), out.ctypes.data, None) == 0
    assert out.tolist() == [10, 0, 16, 10]      # one causal document: 4 x 4 tiles per block, 10 on or below the diagonal
    cost = np.asarray([1, -1, 0, 1], dtype=np.int64)
    ex = np.zeros(4, dtype=np.int32)
    assert lib.hsap_balance(2, cost.ctypes.data, ex.ctypes.data, None) == L.HSAP_ERR_INVALID_ARG   # negative cost
    assert lib.hsap_balance(0, cost.ctypes.data, ex.ctypes.data, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_balance(2, None, ex.ctypes.data, None) == L.HSAP_ERR_INVALID_ARG


def test_executor_struct_layout():
    assert ctypes.sizeof(L.ExecInfo) == 72


def test_executor_validates_before_touching_the_device():
    lib = L.lib()
    good = L.attn_desc(L.shard_desc(2048, 2, "contiguous", 0, 128, 128), 4, 4, 128, 0.1)
    h = ctypes.c_void_p(123)
    # no output pointer, a malformed shard, an unsupported head_dim, unknown options, a bad split
    assert lib.hsap_executor_create(ctypes.byref(good), 0, -1, None) == L.HSAP_ERR_INVALID_ARG
    bad_shard = L.attn_desc(L.shard_desc(2047, 2, "contiguous", 0, 128, 128), 4, 4, 128, 0.1)
    assert lib.hsap_executor_create(ctypes.byref(bad_shard), 0, -1, ctypes.byref(h)) == L.HSAP_ERR_INVALID_ARG
    assert h.value is None                                   # *out cleared on failure
    bad_d = L.attn_desc(L.shard_desc(2048, 2, "contiguous", 0, 128, 128), 4, 4, 96, 0.1)
    assert lib.hsap_executor_create(ctypes.byref(bad_d), 0, -1, ctypes.byref(h)) == L.HSAP_ERR_UNSUPPORTED
    assert lib.hsap_executor_create(ctypes.byref(good), 4, -1, ctypes.byref(h)) == L.HSAP_ERR_INVALID_ARG
    # the backward option needs backward kernels for the shape: refused at creation, before any allocation
    no_bwd = L.attn_desc(L.shard_desc(2048, 2, "contiguous", 0, 128, 128), 4, 4, 64, 0.1)
    assert lib.hsap_executor_create(ctypes.byref(no_bwd), L.EXEC_BACKWARD, -1, ctypes.byref(h)) == \
        L.HSAP_ERR_UNSUPPORTED
    assert "backward" in lib.hsap_last_error().decode()
    assert lib.hsap_fwd_resident_workgroups(ctypes.byref(good), None) == L.HSAP_ERR_INVALID_ARG
    out = ctypes.c_int32(7)
    assert lib.hsap_fwd_resident_workgroups(ctypes.byref(bad_d), ctypes.byref(out)) == L.HSAP_ERR_UNSUPPORTED
    assert out.value == 0
    assert lib.hsap_executor_create(ctypes.byref(good), 0, -2, ctypes.byref(h)) == L.HSAP_ERR_INVALID_ARG
    # calls on a NULL executor
    cu = np.asarray([0, 2048], dtype=np.int32)
    assert lib.hsap_executor_plan(None, cu.ctypes.data, 1, None) == L.HSAP_ERR_INVALID_ARG
    info = L.ExecInfo()
    assert lib.hsap_executor_info(None, ctypes.byref(info)) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_executor_forward(None, 1, 1, 1, 0, 1, 1, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_executor_backward(None, 1, 1, 1, 1, 1, 1, 1, 1, 1, None) == L.HSAP_ERR_INVALID_ARG
    lib.hsap_executor_destroy(None)                          # no-op
    assert lib.hsap_executor_partial_forward(None, 1, 1, 1, 1, 1, None) == L.HSAP_ERR_INVALID_ARG
    assert lib.hsap_executor_merge(None, 1, 1, None) == L.HSAP_ERR_INVALID_ARG
