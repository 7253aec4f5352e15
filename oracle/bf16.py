"""bfloat16 storage rounding for the oracle (test infrastructure only).

bfloat16 keeps the sign, the 8 exponent bits and the top 7 mantissa bits of a
binary32 value.  Rounding is to nearest, ties to even, on the 16 discarded
bits; NaN is kept as a quiet NaN.  Values are returned widened back to
float32 so that NumPy can compute with them exactly.
"""

import numpy as np


def round_bf16(a) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), as float32."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    out = r.astype(np.uint32).view(np.float32).reshape(a32.shape)
    nan = np.isnan(a32)
    if nan.any():
        out = np.where(nan, np.float32(np.nan), out)
    return out
