"""Decoding of an fp8 KV cache.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper treats KV quantization as orthogonal to its selection: a lower
bit-width per cached entry can be stacked on top of it for further bandwidth
savings (section 6, "KV quantization for LLM").  The library's fp8 mode
stores every K and V element as one byte in the OCP 8-bit floating-point
format E4M3 (the "FN" variant: no infinities) and keeps one fp32 scale per
(request, KV head) for K and one for V; the cached value is
``code_value * scale``.

E4M3 as the OCP specification defines it, for a byte ``s eeee mmm``:

* exponent field ``e`` in 1..15: ``(-1)^s * 2^(e - 7) * (1 + m / 8)``;
* ``e = 0`` (subnormal): ``(-1)^s * 2^(-6) * (m / 8)``;
* ``e = 15, m = 7``: NaN (both signs); there are no infinities, so the
  largest finite magnitude is ``2^8 * 1.75 = 448``.

Every such value is exact in fp64, so the oracle dequantizes exactly and then
runs the same fp64 attention as for bf16 caches.
"""

from __future__ import annotations

import numpy as np


def decode_e4m3(codes) -> np.ndarray:
    """fp64 value of every E4M3 byte in ``codes`` (any integer array)."""
    c = np.asarray(codes).astype(np.int64) & 0xFF
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    normal = np.ldexp(1.0 + m / 8.0, (e - 7).astype(np.int64))
    sub = np.ldexp(m / 8.0, -6)
    out = sign * np.where(e == 0, sub, normal)
    return np.where((e == 15) & (c & 0x7 == 7), np.nan, out)


def dequantize(codes, scale) -> np.ndarray:
    """Cached values of one (request, KV head): codes times its scale."""
    return decode_e4m3(codes) * float(scale)
