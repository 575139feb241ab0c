"""Storage formats of the compressed cache (oracle side).

The paper fixes no precision (it only says sink tokens are kept "in full
precision", Section 3.1.1).  The stored state is therefore given in one of two
formats: fp32, or bf16 (8 significant bits, fp32 exponent range).  The oracle
always computes in float64 on the stored values, which float64 holds exactly.

Where the decode step itself writes into the cache (the appended coefficient
row of Section 3.2.1) the value is rounded to the storage format the way a
kernel with an fp32 result register would: float64 -> fp32 (round to nearest
even) -> bf16 (round to nearest even).
"""

import numpy as np

FP32 = "fp32"
BF16 = "bf16"


def to_fp32(x):
    """Round float64 values to fp32 (nearest even) and return them as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def to_bf16(x):
    """Round float64 values to bf16 (via fp32, nearest even on both steps).

    bf16 keeps the upper 16 bits of an fp32 word; rounding adds half an ulp of
    the kept part plus the parity bit of its last kept bit, then truncates.
    NaN/inf do not occur in the oracle's inputs.
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def round_to(x, dtype):
    if dtype == BF16:
        return to_bf16(x)
    if dtype == FP32:
        return to_fp32(x)
    raise ValueError(f"unknown storage dtype {dtype!r}")
