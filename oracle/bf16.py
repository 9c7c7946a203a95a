"""bfloat16 operand emulation for the bf16-GEMM workloads.

A value is first rounded to float32 (the precision in which the device holds
it), then to bfloat16 by round-to-nearest, ties-to-even on the upper 16 bits.
The result is returned as float64 so the oracle keeps computing in float64.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    r = r.astype(np.uint32)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = np.uint32(0x7FC00000)
    return r.view(np.float32).astype(np.float64)


def identity(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)
