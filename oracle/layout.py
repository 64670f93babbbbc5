"""Oracle packer and unpacker of the packed weight layout (test infrastructure).

The paper fixes no bit layout for its formats (the layout figure, Figure 3b,
is absent), so the library defines one; this module restates it from its
definition, bit by bit, with no shared code.

Layout of an n x k matrix, b-bit codes, groups of g along k, kind uniform or
codebook; k % 128 == 0, C = k / 128 chunks per row, G = k / g groups per row.

Codes region (offset 0, n*k*b/8 bytes). A chunk is 128 consecutive codes of one
row, stored in 16*b bytes. Chunk c of row n is split into b slices of 16 bytes;
slice s holds chunk bytes [16s, 16s+16) and lives at byte offset
((n*b + s)*C + c)*16. Chunk bit p is bit (p mod 8) of chunk byte p // 8
(little-endian). Inside a chunk:

  b = 4: code i occupies chunk bits 4i .. 4i+3 (LSB first).
  b = 3: chunk byte j (0..47) has an A field (bits 0-2), a B field (bits 3-5)
         and a 2-bit spare field (bits 6-7).
           code i,      i in [0, 48)  : A field of byte i
           code 48 + j, j in [0, 48)  : B field of byte j
           code 96 + m, m in [0, 32)  : bits 0-1 in the spare field of byte m,
                                        bit 2 in bit 6 + m // 16 of byte 32 + m % 16

Metadata region (offset n*k*b/8):
  uniform : 4 bytes per (row, group) at (n*G + j)*4: binary16 scale in the low
            half, binary16 zero-point (an integer in [0, 2^b)) in the high half.
  codebook: 2^b binary16 entries per (row, group) at (n*G + j)*2^b*2, entry e at +2e.
"""
from __future__ import annotations

import numpy as np

UNIFORM, CODEBOOK = 0, 1
CHUNK = 128


def chunk_bit_positions(bits: int) -> np.ndarray:
    """pos[i, t] = chunk bit that holds bit t of code i (i < 128, t < bits)."""
    pos = np.full((CHUNK, bits), -1, dtype=np.int64)
    for i in range(CHUNK):
        for t in range(bits):
            if bits == 4:
                pos[i, t] = 4 * i + t
            elif bits == 3:
                if i < 48:
                    pos[i, t] = 8 * i + t
                elif i < 96:
                    pos[i, t] = 8 * (i - 48) + 3 + t
                else:
                    m = i - 96
                    if t < 2:
                        pos[i, t] = 8 * m + 6 + t
                    else:
                        pos[i, t] = 8 * (32 + m % 16) + 6 + m // 16
            else:
                raise ValueError(f"unsupported bits {bits}")
    return pos


def _meta_bytes_per_group(bits: int, kind: int) -> int:
    return 4 if kind == UNIFORM else 2 * (1 << bits)


def _check(n, k, bits, group, kind):
    if bits not in (3, 4) or kind not in (UNIFORM, CODEBOOK):
        raise ValueError("bits must be 3 or 4, kind uniform (0) or codebook (1)")
    if n < 0 or k <= 0 or k % CHUNK or group <= 0 or k % group or CHUNK % group and group % CHUNK:
        raise ValueError("k must be a positive multiple of 128 and of the group size")


def pack_code_region(codes, bits) -> np.ndarray:
    """Codes region (uint8, n*k*b/8 bytes) of codes [n][k]."""
    codes = np.asarray(codes, dtype=np.uint8)
    n, k = codes.shape
    if np.any(codes >= (1 << bits)):
        raise ValueError("code out of range")
    C = k // CHUNK
    pos = chunk_bit_positions(bits)
    chunks = codes.reshape(n, C, CHUNK)
    bitarr = np.zeros((n, C, CHUNK * bits), dtype=np.uint8)
    for i in range(CHUNK):
        for t in range(bits):
            bitarr[:, :, pos[i, t]] = (chunks[:, :, i] >> t) & 1
    chunk_bytes = np.packbits(bitarr, axis=-1, bitorder="little")          # [n, C, 16b]
    planes = chunk_bytes.reshape(n, C, bits, 16).transpose(0, 2, 1, 3)      # [n, b, C, 16]
    return np.ascontiguousarray(planes).reshape(-1)


def unpack_code_region(blob, n, k, bits) -> np.ndarray:
    """Codes [n][k] (uint8) from the first n*k*b/8 bytes of a blob."""
    blob = np.asarray(blob, dtype=np.uint8).reshape(-1)
    C = k // CHUNK
    ncode = n * k * bits // 8
    planes = blob[:ncode].reshape(n, bits, C, 16).transpose(0, 2, 1, 3)   # [n, C, b, 16]
    chunk_bytes = np.ascontiguousarray(planes).reshape(n, C, 16 * bits)
    bitarr = np.unpackbits(chunk_bytes, axis=-1, bitorder="little")       # [n, C, 128b]
    pos = chunk_bit_positions(bits)
    codes = np.zeros((n, C, CHUNK), dtype=np.uint8)
    for i in range(CHUNK):
        for t in range(bits):
            codes[:, :, i] |= bitarr[:, :, pos[i, t]] << t
    return codes.reshape(n, k)


def pack(codes, bits, group, kind, scales=None, zeros=None, codebook=None) -> np.ndarray:
    """Packed blob (uint8) of codes [n][k] and the per-group tables (binary16 bit patterns)."""
    codes = np.asarray(codes, dtype=np.uint8)
    n, k = codes.shape
    _check(n, k, bits, group, kind)
    G = k // group
    code_region = pack_code_region(codes, bits)
    if kind == UNIFORM:
        s = np.asarray(scales, dtype=np.uint16).reshape(n, G).astype(np.uint32)
        z = np.asarray(zeros, dtype=np.uint16).reshape(n, G).astype(np.uint32)
        meta = (s | (z << 16)).astype("<u4").view(np.uint8).reshape(-1)
    else:
        cb = np.asarray(codebook, dtype=np.uint16).reshape(n, G, 1 << bits)
        meta = cb.astype("<u2").view(np.uint8).reshape(-1)
    return np.concatenate([code_region, meta])


def unpack(blob, n, k, bits, group, kind):
    """Inverse of :func:`pack`: (codes [n][k] uint8, tables) from a packed blob.

    Returns (codes, scales, zeros, None) for uniform and (codes, None, None,
    codebook) for codebook; tables are binary16 bit patterns (uint16).
    """
    _check(n, k, bits, group, kind)
    blob = np.asarray(blob, dtype=np.uint8).reshape(-1)
    G = k // group
    ncode = n * k * bits // 8
    codes = unpack_code_region(blob, n, k, bits)
    meta = blob[ncode:ncode + n * G * _meta_bytes_per_group(bits, kind)]
    if kind == UNIFORM:
        words = meta.view("<u4").reshape(n, G)
        return codes, (words & 0xFFFF).astype(np.uint16), (words >> 16).astype(np.uint16), None
    cb = meta.view("<u2").reshape(n, G, 1 << bits).astype(np.uint16)
    return codes, None, None, cb
