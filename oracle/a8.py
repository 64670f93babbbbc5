"""Oracle of the 8-bit-activation path (test infrastructure).

The paper quantizes activations to 8 bits and not below (Section 2.4), and its
W3A8G128 configurations (Table 1) and all of Table 2 use 8-bit round-to-nearest
per-token activations. Per token here means per activation vector: one
symmetric scale for the whole vector.

  amax  = max_k |x[k]|                 (x binary16, exact)
  inv   = fp32(127 / amax),  s_x = fp32(amax / 127)       (amax = 0: xq = 0, s_x = 0)
  xq[k] = clamp(RNE(x[k] * inv), -127, 127)                int8, the product exact
  y[n]  = s_x * sum_j s[n,j] * sum_{k in group j} (q[n,k] - z[n,j]) * xq[k]

Q4X with 8-bit activations (the paper's Table 2 runs Q4X with 8-bit RTN per-token
activations): the same xq and s_x, and the fp16 entries of the selected
sub-codebook in place of the integer levels,
  y[n]  = s_x * sum_j s[n,j] * sum_{k in group j} CB[t[n,j]][q[n,k]] * xq[k]
(the group scale multiplies the group's sum: the exact products s * CB, not W'
rounded to binary16).

Per-group codebooks with 8-bit activations (QuantX picks uniform or non-uniform
groups per layer, Section 2.2, and runs its W3A8 configurations, Table 1, with
either): the same xq and s_x, and the group's fp16 table entries, which are W'
exactly,
  y[n]  = s_x * sum_k C[n, j(k)][q[n,k]] * xq[k]          (j(k) = k // g).

The steps that decide an integer are the ones the GPU takes: the fp32 scale
inv, and the nearest integer to the exact product of a binary16 x and the fp32
inv (at most 35 significant bits, exact in fp64 here; one fused multiply-add
with a rounding constant there), so both sides reach the same int8 codes; the
sums are exact integers and the scaling is done in fp64 here. The weights
enter as the exact s * (q - z) of each uniform level (the integer product path
never rounds W' to binary16).
"""
from __future__ import annotations

import numpy as np


def quantize_activation(x16) -> tuple:
    """(xq int8 [k], s_x float32) of one binary16 activation vector."""
    x = np.asarray(x16, dtype=np.float16).astype(np.float32)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    if amax == 0:
        return np.zeros(x.shape, np.int8), np.float32(0)
    inv = np.float32(np.float32(127.0) / amax)
    s_x = np.float32(amax / np.float32(127.0))
    q = np.rint(x.astype(np.float64) * np.float64(inv))  # exact product, then nearest-even
    return np.clip(q, -127, 127).astype(np.int8), s_x


def gemv_a8(codes, group, scales, zeros, x16) -> np.ndarray:
    """fp64 y [n] of uniform codes [n][k] (binary16 scales/zeros [n][k/g]) and fp16 x [k]."""
    codes = np.asarray(codes).astype(np.int64)
    n, k = codes.shape
    G = k // group
    xq, s_x = quantize_activation(x16)
    s = np.asarray(scales, np.uint16).reshape(n, G).view(np.float16).astype(np.float64)
    z = np.asarray(zeros, np.uint16).reshape(n, G).view(np.float16).astype(np.int64)
    j = np.arange(k) // group
    d = codes - z[:, j]                                     # exact integers
    per_group = np.zeros((n, G), dtype=np.int64)
    prod = d * xq.astype(np.int64)[None, :]
    for g in range(G):
        per_group[:, g] = prod[:, g * group:(g + 1) * group].sum(axis=1)
    return float(s_x) * (s * per_group.astype(np.float64)).sum(axis=1)


def gemv_a8_q4x(codes, scales, selectors, codebook, x16) -> np.ndarray:
    """fp64 y [n] of a Q4X matrix (codes [n][k], binary16 scales [n][k/64], selectors
    [n][k/64], binary16 codebook [4][16]) and fp16 x [k] quantized to 8 bits."""
    codes = np.asarray(codes).astype(np.int64)
    n, k = codes.shape
    G = k // 64
    xq, s_x = quantize_activation(x16)
    s = np.asarray(scales, np.uint16).reshape(n, G).view(np.float16).astype(np.float64)
    t = np.asarray(selectors).reshape(n, G).astype(np.int64)
    cb = np.asarray(codebook, np.uint16).reshape(4, 16).view(np.float16).astype(np.float64)
    j = np.arange(k) // 64
    entries = cb[t[:, j], codes]                              # CB[t][q], exact binary16 values
    prod = entries * xq.astype(np.float64)[None, :]
    per_group = prod.reshape(n, G, 64).sum(axis=2)
    return float(s_x) * (s * per_group).sum(axis=1)


def gemv_a8_codebook(codes, group, codebook, x16) -> np.ndarray:
    """fp64 y [n] of per-group codebook codes [n][k] (binary16 tables [n][k/g][2^b])
    and fp16 x [k] quantized to 8 bits."""
    codes = np.asarray(codes).astype(np.int64)
    n, k = codes.shape
    G = k // group
    xq, s_x = quantize_activation(x16)
    E = np.asarray(codebook).shape[-1]
    cb = np.asarray(codebook, np.uint16).reshape(n, G, E).view(np.float16).astype(np.float64)
    j = np.arange(k) // group
    entries = cb[np.arange(n)[:, None], j[None, :], codes]   # C[n, j(k)][q], exact binary16 values
    return float(s_x) * (entries * xq.astype(np.float64)[None, :]).sum(axis=1)
