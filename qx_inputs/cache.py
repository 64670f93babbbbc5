"""Disk cache of quantized synthetic matrices (input preparation only).

Generating and quantizing the 224 matrices of the 7B decode step takes about 20 s
of host time, and the GPU tests and the benchmark each need them. A quantized
matrix is stored here once, keyed by everything that determines it: the matrix
spec (name, shape, distribution, seed, stream, format), the row range, a format
version, and a hash of the quantizer sources. Arrays are written with numpy's
.npy format and read back with allow_pickle=False.

Location: $QX_QUANT_CACHE (default /tmp/qx_quant_cache); "off" disables it.
Budget: $QX_QUANT_CACHE_GB (default 12) gigabytes; a matrix that would exceed it
is not stored. Any I/O error simply falls back to quantizing.
"""
from __future__ import annotations

import hashlib
import os
from typing import Optional

import numpy as np

FORMAT_VERSION = 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_FIELDS = ("codes", "scales", "zeros", "codebook", "selectors")
_src_hash = None


def _sources_hash() -> str:
    global _src_hash
    if _src_hash is None:
        h = hashlib.sha256()
        for f in ("_gen.cpp", "__init__.py", "q4x.py"):
            with open(os.path.join(_HERE, f), "rb") as fh:
                h.update(fh.read())
        _src_hash = h.hexdigest()[:16]
    return _src_hash


def cache_dir() -> Optional[str]:
    d = os.environ.get("QX_QUANT_CACHE", "/tmp/qx_quant_cache")
    return None if d.lower() in ("", "off", "0", "none") else d


def key(spec, row0: int, rows: Optional[int]) -> str:
    desc = (f"v{FORMAT_VERSION}|{_sources_hash()}|{spec.name}|{spec.n}x{spec.k}|{spec.dist}|{spec.p!r}|"
            f"{spec.seed}|{spec.stream}|{spec.bits}|{spec.group}|{spec.kind}|{row0}|{rows}")
    return hashlib.sha256(desc.encode()).hexdigest()[:32]


def _dir_bytes(d: str) -> int:
    total = 0
    for root, _, files in os.walk(d):
        for f in files:
            try:
                total += os.path.getsize(os.path.join(root, f))
            except OSError:
                pass
    return total


def load(spec, row0: int, rows: Optional[int]):
    """The cached QuantWeight, or None."""
    from . import QuantWeight
    d = cache_dir()
    if d is None:
        return None
    path = os.path.join(d, key(spec, row0, rows))
    if not os.path.exists(os.path.join(path, "done")):
        return None
    try:
        arrays = {}
        for f in _FIELDS:
            p = os.path.join(path, f + ".npy")
            arrays[f] = np.load(p, allow_pickle=False) if os.path.exists(p) else None
        n = arrays["codes"].shape[0]
        return QuantWeight(n, spec.k, spec.bits, spec.group, spec.kind, arrays["codes"], arrays["scales"],
                           arrays["zeros"], arrays["codebook"], selectors=arrays["selectors"])
    except (OSError, ValueError):
        return None


def store(spec, row0: int, rows: Optional[int], q) -> bool:
    """Write q unless the cache is off or its budget would be exceeded; True if stored."""
    d = cache_dir()
    if d is None:
        return False
    budget = float(os.environ.get("QX_QUANT_CACHE_GB", "12")) * 1e9
    size = sum(getattr(q, f).nbytes for f in _FIELDS if getattr(q, f) is not None)
    path = os.path.join(d, key(spec, row0, rows))
    tmp = f"{path}.tmp{os.getpid()}"
    try:
        os.makedirs(d, exist_ok=True)
        if _dir_bytes(d) + size > budget:
            return False
        os.makedirs(tmp, exist_ok=True)
        for f in _FIELDS:
            a = getattr(q, f)
            if a is not None:
                np.save(os.path.join(tmp, f + ".npy"), np.ascontiguousarray(a), allow_pickle=False)
        open(os.path.join(tmp, "done"), "w").close()
        os.replace(tmp, path)
        return True
    except OSError:
        import shutil
        shutil.rmtree(tmp, ignore_errors=True)
        return False
