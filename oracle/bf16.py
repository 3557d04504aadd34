"""bfloat16 operand rounding for the oracle's bf16-MFMA mode.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The bf16 mode of the stage rounds every operand of a contraction (weights from
the fp32 master copy, activations, upstream gradients) to bfloat16 with
round-to-nearest-even and accumulates in higher precision; everything else
stays fp32.  bfloat16 is the upper half of an IEEE-754 binary32: 1 sign bit,
8 exponent bits, 7 stored mantissa bits.  Rounding to nearest-even on the
16 discarded bits is the textbook rule: add 0x7FFF plus the lowest kept bit,
then truncate.  Values are first rounded to binary32, as the device holds
them.
"""
from __future__ import annotations

import numpy as np


def round_bf16(a) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even); returns float64 values."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    out = r.astype(np.uint32).view(np.float32)
    # NaN stays NaN (none occur for finite inputs in this code base)
    nan = np.isnan(f)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.astype(np.float64).reshape(np.shape(a))
