"""Sizes and bits-per-weight (test infrastructure).

The paper reports bits per weight (BPW) including per-group metadata, e.g. a
legacy 4-bit format packs 32 weights and an fp16 scale into 18 bytes (4.5 BPW)
and its own 4-bit format stores a 2-byte scale, a 2-bit codebook selector and
64 4-bit indices per group of 64 (4.28 BPW), Section 3.2.
"""
from __future__ import annotations

from .layout import UNIFORM


def packed_size(n: int, k: int, bits: int, group: int, kind: int) -> int:
    """Bytes of the packed blob: codes plus per-group tables."""
    meta = 4 if kind == UNIFORM else 2 * (1 << bits)
    return n * k * bits // 8 + n * (k // group) * meta


def bits_per_weight(bits: int, group: int, meta_bits_per_group: int) -> float:
    """Code bits plus metadata bits spread over the group."""
    return bits + meta_bits_per_group / group
