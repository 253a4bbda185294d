"""Operand rounding of the bf16 variant of the dense products.

The variant (a precision option of the dense transforms, Section 4.3's
products computed on matrix units) rounds each operand of a product to
bfloat16 -- 1 sign bit, 8 exponent bits, 7 stored fraction bits -- with
round to nearest, ties to even, and multiplies and accumulates in float32
or wider. The oracle models it by rounding operands here and multiplying in
float64.
"""
import numpy as np


def round_bf16(x):
    """float32 values rounded to the nearest bfloat16 (ties to even),
    returned as float64. NaN stays NaN; magnitudes that round past the
    largest finite bfloat16 become infinite."""
    a = np.asarray(x, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    # add half a bfloat16 unit, minus one unless the kept last bit is odd:
    # exact halves then round to the even neighbour
    kept_lsb = (u >> 16) & 1
    r = (((u + 0x7FFF + kept_lsb) >> 16) << 16).astype(np.uint32)
    out = r.view(np.float32)
    out = np.where(np.isnan(a), a, out)
    return out.astype(np.float64)
