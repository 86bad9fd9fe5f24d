"""bf16 emulation for the oracle (fp64 arithmetic).

The bf16 workloads round GEMM inputs, q/k/v and the KV cache to bf16 with
round-to-nearest-even; everything else is carried in fp64 here.  bf16 has 8
significant bits (1 implicit + 7 stored), so rounding a finite, normal x is
``ldexp(round_half_even(m * 2**8), e - 8)`` with ``x = m * 2**e``,
``0.5 <= |m| < 1``.  (The tests pin this against exhaustive bf16 enumeration.)
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value (ties to even); returns fp64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    r = np.round(m * 256.0)            # numpy rounds halves to even
    return np.ldexp(r / 256.0, e)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode uint16 bf16 bit patterns to fp64 (bf16 is the top half of an fp32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def to_f64(w: np.ndarray) -> np.ndarray:
    """Weights as stored by the workload generator (uint16 bf16 bits or fp32) -> fp64."""
    if w.dtype == np.uint16:
        return bf16_bits_to_f64(w)
    return np.asarray(w, dtype=np.float64)
