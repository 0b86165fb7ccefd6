"""Storage rounding used by the oracle's precision-emulation modes.

Test infrastructure only (see ``oracle/__init__.py``).

The paper states no numeric precision.  The oracle computes in float64; in
its emulation modes it rounds values to the storage type at exactly the points
where the GPU path stores them (bfloat16 or float32), keeping float64
arithmetic everywhere else.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (8 significant
    bits, ties to even), directly from float64 (no intermediate float32, so
    no double rounding).  Result is float64.  Overflow/subnormal ranges are
    not needed by the workloads and are not treated specially."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                  # x = m * 2**e, 0.5 <= |m| < 1
    q = np.rint(m * 256.0)              # 8 significant bits, half-to-even
    return np.ldexp(q, e - 8)


def round_f32(x) -> np.ndarray:
    """Round float64 values to float32 (IEEE round to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def identity(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


ROUNDERS = {"f64": identity, "f32": round_f32, "bf16": round_bf16}
