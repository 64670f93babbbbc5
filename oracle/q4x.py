"""Oracle of the Q4X format (test infrastructure).

Q4X is the paper's codebook format for 4-bit weights (Section 3.2, the Q4X item;
Figure 3a/3b captions): a matrix carries one codebook of 64 binary16 centroids,
made of 4 sub-codebooks of 16 (one per learned histogram), and every group of
64 consecutive weights of a row stores a binary16 scale, a 2-bit selector that
names its sub-codebook and 64 4-bit centroid indices, 4 + 18/64 = 4.28 bits per
weight. A weight is the scaled centroid,

  W'[n,k] = fp16_RNE( s[n,j] * CB[sel[n,j]][q[n,k]] ),   j = k // 64,

the product of two binary16 values taken exactly in fp64 (at most 22
significant bits) and rounded once, as for the uniform groups.

Packed layout (Q4X; k a multiple of 128, G = k/64 groups and W = ceil(G/16)
selector words per row); the paper fixes no byte layout, so the library
defines this one:
  codes     offset 0, n*k/2 bytes: the 4-bit codes region of the general layout
  scales    offset S0 = n*k/2: binary16 per (row, group) at S0 + (n*G + j)*2
  selectors offset L0 = S0 + n*G*2: W little-endian uint32 words per row; the
            selector of group j is bits 2*(j%16), 2*(j%16)+1 of word
            L0 + (n*W + j//16)*4; unused bits are zero
  codebook  offset B0 = L0 + n*W*4 rounded up to a multiple of 16: 64 binary16,
            entry e of sub-codebook t at B0 + (16*t + e)*2
"""
from __future__ import annotations

import numpy as np

from .layout import CHUNK, pack_code_region, unpack_code_region

GROUP = 64
SUBBOOKS, ENTRIES = 4, 16


def _dims(n: int, k: int):
    if n < 0 or k <= 0 or k % CHUNK:
        raise ValueError("k must be a positive multiple of 128")
    G = k // GROUP
    W = (G + 15) // 16
    s0 = n * k // 2
    l0 = s0 + n * G * 2
    b0 = (l0 + n * W * 4 + 15) // 16 * 16
    return G, W, s0, l0, b0


def packed_size(n: int, k: int) -> int:
    """Bytes of a Q4X blob: codes, scales, selector words, padding, 64-entry codebook."""
    return _dims(n, k)[4] + SUBBOOKS * ENTRIES * 2


def pack(codes, scales, selectors, codebook) -> np.ndarray:
    """Q4X blob (uint8) of codes [n][k] (< 16), scales [n][G] (binary16 bits),
    selectors [n][G] (< 4) and the codebook [4][16] (binary16 bits)."""
    codes = np.asarray(codes, dtype=np.uint8)
    n, k = codes.shape
    G, W, s0, l0, b0 = _dims(n, k)
    sel = np.asarray(selectors, dtype=np.uint8).reshape(n, G)
    if np.any(sel >= SUBBOOKS):
        raise ValueError("selector out of range")
    blob = np.zeros(packed_size(n, k), dtype=np.uint8)
    blob[:s0] = pack_code_region(codes, 4)
    blob[s0:l0] = np.asarray(scales, np.uint16).reshape(n, G).astype("<u2").view(np.uint8).reshape(-1)
    words = np.zeros((n, W), dtype=np.uint64)
    for j in range(G):
        words[:, j // 16] |= sel[:, j].astype(np.uint64) << np.uint64(2 * (j % 16))
    blob[l0:l0 + n * W * 4] = words.astype("<u4").view(np.uint8).reshape(-1)
    cb = np.asarray(codebook, np.uint16).reshape(SUBBOOKS * ENTRIES)
    blob[b0:] = cb.astype("<u2").view(np.uint8)
    return blob


def unpack(blob, n: int, k: int):
    """Inverse of :func:`pack`: (codes, scales, selectors, codebook)."""
    blob = np.asarray(blob, dtype=np.uint8).reshape(-1)
    G, W, s0, l0, b0 = _dims(n, k)
    codes = unpack_code_region(blob, n, k, 4)
    scales = blob[s0:l0].view("<u2").reshape(n, G).astype(np.uint16)
    words = blob[l0:l0 + n * W * 4].view("<u4").reshape(n, W).astype(np.uint64)
    sel = np.empty((n, G), dtype=np.uint8)
    for j in range(G):
        sel[:, j] = (words[:, j // 16] >> np.uint64(2 * (j % 16))) & np.uint64(3)
    cb = blob[b0:b0 + SUBBOOKS * ENTRIES * 2].view("<u2").reshape(SUBBOOKS, ENTRIES).astype(np.uint16)
    return codes, scales, sel, cb


def dequant(codes, scales, selectors, codebook) -> np.ndarray:
    """fp16 W' [n][k] = fp16_RNE(s * CB[sel][q]) per weight (exact product in fp64)."""
    codes = np.asarray(codes)
    n, k = codes.shape
    G = k // GROUP
    j = np.arange(k) // GROUP
    s = np.asarray(scales, np.uint16).reshape(n, G).view(np.float16).astype(np.float64)
    sel = np.asarray(selectors).reshape(n, G).astype(np.int64)
    cb = np.asarray(codebook, np.uint16).reshape(SUBBOOKS, ENTRIES).view(np.float16).astype(np.float64)
    centroid = cb[sel[:, j], codes.astype(np.int64)]
    with np.errstate(over="ignore"):  # products past the binary16 range round to +-inf
        return (s[:, j] * centroid).astype(np.float16)


def dequant_packed(blob, n: int, k: int) -> np.ndarray:
    return dequant(*unpack(blob, n, k))
