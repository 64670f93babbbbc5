"""Oracle products in fp64 and the error metric (test infrastructure).

Decoding multiplies each dequantized weight matrix by one 16-bit activation
vector (batch-1 GEMV, the memory-bound case of Section 2.4); prefill multiplies
it by an activation matrix. Both are evaluated here in fp64 on the fp16 values
of W', x and X, so the only rounding is fp64's, far below the fp32 accumulate
of the GPU path.
"""
from __future__ import annotations

import numpy as np


def gemv(w16: np.ndarray, x16: np.ndarray) -> np.ndarray:
    """y[n] = sum_k W'[n,k] x[k] in fp64."""
    return np.asarray(w16, np.float64) @ np.asarray(x16, np.float64)


def gemm(x16: np.ndarray, w16: np.ndarray) -> np.ndarray:
    """Y[m,n] = sum_k X[m,k] W'[n,k] in fp64."""
    return np.asarray(x16, np.float64) @ np.asarray(w16, np.float64).T


def normwise_rel_err(y, y_ref) -> float:
    """max_i |y_i - yref_i| / max_i |yref_i| over one output vector (0 if both vanish)."""
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    den = float(np.max(np.abs(y_ref))) if y_ref.size else 0.0
    num = float(np.max(np.abs(y - y_ref))) if y_ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den
