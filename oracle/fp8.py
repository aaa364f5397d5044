"""fp8 (e4m3) quantisation of Q and K for the fp8 score variant.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper computes attention in bf16; the fp8 QK variant is this build's
extension (scores from fp8 operands, the rest unchanged).  What it computes
is fixed here, and the variant's attention is then the oracle's attention on
the dequantised values:

* Per group g and head h of x [G, rows, H, d] (a shard's Q: G = 1; the
  chunks' K: G = P): amax = max |x| over rows and d, in fp32.
* scale = amax / 448 and inv = 448 / amax, each one fp32 division (both 0
  when amax = 0).  448 is the largest finite e4m3 value.
* code = e4m3(clamp(x * inv, -448, 448)): fp32 product, clamp, then round to
  nearest even into e4m3 (OCP "fn" format: 4 exponent bits, bias 7, no
  infinities).  The rounding step is torch's float8_e4m3fn conversion.
* dequantised value = decode(code) * scale.

Pins (``tests/test_oracle_pins.py``): hand-computed codes of a worked
example, amax elements landing on +-448, the round-trip bound of half an e4m3
step, and decode(code) equal to the value it encodes for every code.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np
import torch

E4M3_MAX = np.float32(448.0)


def quantize_fp8(x) -> Tuple[np.ndarray, np.ndarray]:
    """(codes uint8 [G, rows, H, d], scale float32 [G, H]) of x [G, rows, H, d]."""
    xf = np.asarray(x, dtype=np.float32)
    amax = np.abs(xf).max(axis=(1, 3)).astype(np.float32)
    safe = np.where(amax > 0, amax, np.float32(1))
    inv = np.where(amax > 0, E4M3_MAX / safe, np.float32(0)).astype(np.float32)
    scale = np.where(amax > 0, safe / E4M3_MAX, np.float32(0)).astype(np.float32)
    y = np.clip(xf * inv[:, None, :, None], -E4M3_MAX, E4M3_MAX).astype(np.float32)
    codes = torch.from_numpy(np.ascontiguousarray(y)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes, scale


def decode_fp8(codes) -> np.ndarray:
    """The e4m3 values of ``codes`` (float64)."""
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(codes, dtype=np.uint8))).view(torch.float8_e4m3fn)
    return t.to(torch.float64).numpy()


def dequantize_fp8(codes, scale) -> np.ndarray:
    """decode(code) * scale[g, h], float64 [G, rows, H, d]."""
    return decode_fp8(codes) * np.asarray(scale, dtype=np.float64)[:, None, :, None]
