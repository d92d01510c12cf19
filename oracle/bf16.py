"""Round-to-nearest-even conversion of float32 values to bfloat16 (oracle side).

TEST INFRASTRUCTURE ONLY (see ``oracle/ir.py``).

bfloat16 keeps the sign, the 8 exponent bits and the top 7 mantissa bits of a
float32. Rounding to nearest, ties to even, of the 32-bit pattern ``u`` is:
add ``0x7FFF`` plus the lowest kept bit ``(u >> 16) & 1`` and truncate the low
16 bits. Overflow carries into the exponent and yields infinity, as it should.
NaN inputs stay NaN (a quiet NaN). This is the ``dataTypeCast`` of Table 1
applied from f32 to bf16; the paper fixes no rounding mode, and
round-to-nearest-even is the IEEE default.
"""
from __future__ import annotations

import numpy as np


def round_to_bf16(a) -> np.ndarray:
    """Return the bf16 value nearest to each float32 element, as float64."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    r = (r & np.uint64(0xFFFFFFFF)).astype(np.uint32)
    r = np.where(np.isnan(f), np.uint32(0x7FC00000), r)
    return r.view(np.float32).astype(np.float64)


def bf16_bits(a) -> np.ndarray:
    """The 16-bit patterns of ``round_to_bf16(a)`` (for bit-exact comparisons)."""
    v = round_to_bf16(a).astype(np.float32)
    return (v.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
