"""Oracle dequantization (test infrastructure).

Uniform groups use equally spaced levels and codebook groups use a per-group
table of non-uniform levels; the paper keeps both kinds and picks per matrix
(Section 2.2, Figure 2a). Inference turns codes back into 16-bit weights in a
custom dequantization kernel before the product (Section 2.4).

  uniform : W' = fp16_RNE(s * (q - z)), the product taken exactly in fp64
            (|q - z| < 16 and s is binary16, so s*(q-z) has at most 15
            significant bits) and rounded once to binary16 by numpy.
  codebook: W' = C[q], a table lookup with no arithmetic.
"""
from __future__ import annotations

import numpy as np

from .layout import CODEBOOK, UNIFORM, unpack


def dequant(codes, group, kind, scales=None, zeros=None, codebook=None) -> np.ndarray:
    """fp16 W' [n][k] from codes [n][k] and binary16 tables."""
    codes = np.asarray(codes)
    n, k = codes.shape
    G = k // group
    j = np.arange(k) // group
    if kind == UNIFORM:
        s = np.asarray(scales, np.uint16).reshape(n, G).view(np.float16).astype(np.float64)
        z = np.asarray(zeros, np.uint16).reshape(n, G).view(np.float16).astype(np.float64)
        exact = s[:, j] * (codes.astype(np.float64) - z[:, j])
        return exact.astype(np.float16)
    if kind == CODEBOOK:
        E = np.asarray(codebook).shape[-1]
        cb = np.asarray(codebook, np.uint16).reshape(n, G, E).view(np.float16)
        rows = np.arange(n)[:, None]
        return cb[rows, j[None, :], codes.astype(np.int64)]
    raise ValueError("kind must be uniform (0) or codebook (1)")


def dequant_packed(blob, n, k, bits, group, kind) -> np.ndarray:
    """fp16 W' straight from a packed blob (unpack, then dequantize)."""
    codes, s, z, cb = unpack(blob, n, k, bits, group, kind)
    return dequant(codes, group, kind, s, z, cb)
