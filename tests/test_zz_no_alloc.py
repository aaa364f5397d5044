"""The allocation-free quantisation entry point (hsap_quantize_fp8_noalloc) against the entry
point that takes a workspace (hsap_quantize_fp8): codes and scales identical bit for bit (integer
and byte work), on calls in a row that shrink, so the scratch array still holds the previous
call's larger contents when the next one runs.  The first call uses the scratch limit exactly."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2606_30460_amd import _lib as L

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _input(shape, seed):
    g = torch.Generator().manual_seed(seed)
    G, rows, H, d = shape
    x = torch.randn(shape, generator=g) * torch.logspace(-2, 2, H).view(1, 1, H, 1)
    x = x.to(torch.bfloat16)
    x[G // 2, :, H // 2, :] = 0            # a slice with amax 0: scale 0, codes 0
    return x.cuda()


def _quantize_both(x):
    G, rows, H, d = x.shape
    codes_ws = torch.full(x.shape, 0xAB, dtype=torch.uint8, device=x.device)
    scale_ws = torch.full((G, H), float("nan"), dtype=torch.float32, device=x.device)
    work = torch.full((G * H * L.QUANT_SPLIT,), float("nan"), dtype=torch.float32, device=x.device)
    L.quantize_fp8(x, codes_ws, scale_ws, work)
    codes_na = torch.full(x.shape, 0xCD, dtype=torch.uint8, device=x.device)
    scale_na = torch.full((G, H), float("nan"), dtype=torch.float32, device=x.device)
    L.quantize_fp8_noalloc(x, codes_na, scale_na)
    torch.cuda.synchronize()
    return codes_ws.cpu().numpy(), scale_ws.cpu().numpy(), codes_na.cpu().numpy(), scale_na.cpu().numpy()


def test_noalloc_matches_workspace_entry_point():
    shapes = [(64, 16, 64, 16),            # 4096 slices: the scratch limit
              (8, 512, 8, 128),            # 64 slices
              (1, 100, 4, 64)]             # 4 slices
    for i, shape in enumerate(shapes):
        _say("no-alloc quantisation, call", i, "shape", shape)
        x = _input(shape, 100 + i)
        c_ws, s_ws, c_na, s_na = _quantize_both(x)
        assert np.array_equal(c_na, c_ws), shape
        assert np.array_equal(s_na, s_ws), shape
        ref_c, ref_s = oracle.quantize_fp8(x.float().cpu().numpy())
        assert np.array_equal(c_na, ref_c) and np.array_equal(s_na, ref_s), shape


def test_noalloc_rejects_beyond_the_scratch_limit():
    lib = L.lib()
    fake = ctypes.c_void_p(4096)    # never dereferenced: the size check fails first
    st = lib.hsap_quantize_fp8_noalloc(fake, 65, 16, 64, 16, fake, fake, None)   # 4160 slices
    assert st == L.HSAP_ERR_UNSUPPORTED
    assert "4096" in lib.hsap_last_error().decode()
