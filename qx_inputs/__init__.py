"""Seeded synthetic inputs shared by the oracle and the HIP path.

Holds only random draws and input preparation: synthetic fp32 weights with the
per-matrix shapes the paper motivates (narrow, peaked attention weights versus
wider MLP weights, Section 2.1; activation outliers, Section 2.4), and the
group-wise quantizers that turn those weights into the integer codes and fp16
tables that the library's packer takes as input (uniform versus per-group
codebook, Section 2.2). Nothing here unpacks, dequantizes or multiplies.

The native core is ``_gen.cpp`` (Philox4x64-10 counter generator, binary16
rounding, quantizers), built with g++ into ``_libqxinputs.so`` next to it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "_gen.cpp")
_LIB = os.path.join(_HERE, "_libqxinputs.so")

DIST = {"normal": 0, "laplace": 1, "t4": 2}
UNIFORM, CODEBOOK, Q4X = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the native generator with g++ (OpenMP). Returns the .so path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared",
               "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, u64, c_int, dbl = ctypes.c_int64, ctypes.c_uint64, ctypes.c_int, ctypes.c_double
        L.qxi_philox4x64.argtypes = [P, P, P]
        L.qxi_philox4x64.restype = None
        L.qxi_double_to_half.argtypes = [P, i64, c_int, P]
        L.qxi_double_to_half.restype = None
        for name in ("qxi_fill_f64", "qxi_fill_f32"):
            f = getattr(L, name)
            f.argtypes = [c_int, dbl, u64, u64, u64, i64, P, c_int]
            f.restype = c_int
        L.qxi_quantize_uniform.argtypes = [P, i64, i64, c_int, c_int, P, P, P, c_int]
        L.qxi_quantize_uniform.restype = c_int
        L.qxi_quantize_codebook.argtypes = [P, i64, i64, c_int, c_int, c_int, P, P, P, P, c_int]
        L.qxi_quantize_codebook.restype = c_int
        L.qxi_q4x_histograms.argtypes = [P, i64, P, P, c_int]
        L.qxi_q4x_histograms.restype = c_int
        L.qxi_q4x_assign.argtypes = [P, i64, P, P, P, P, c_int]
        L.qxi_q4x_assign.restype = c_int
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, int(os.environ.get("OMP_NUM_THREADS", n))))


# ------------------------------------------------------------------ raw draws
def philox4x64(counter, key) -> np.ndarray:
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.empty(4, dtype=np.uint64)
    lib().qxi_philox4x64(_ptr(c), _ptr(k), _ptr(out))
    return out


def double_to_half_bits(x, mode: int = 0) -> np.ndarray:
    """binary16 bits of float64 values; mode 0 = nearest-even, 1 = toward +inf."""
    a = np.ascontiguousarray(x, dtype=np.float64).ravel()
    out = np.empty(a.size, dtype=np.uint16)
    lib().qxi_double_to_half(_ptr(a), a.size, mode, _ptr(out))
    return out.reshape(np.shape(x))


def fill(dist: str, p: float, seed: int, stream: int, start: int, count: int,
         dtype=np.float64) -> np.ndarray:
    out = np.empty(count, dtype=dtype)
    fn = lib().qxi_fill_f64 if dtype == np.float64 else lib().qxi_fill_f32
    if dtype not in (np.float64, np.float32):
        raise ValueError("dtype must be float64 or float32")
    rc = fn(DIST[dist], float(p), seed, stream, start, count, _ptr(out), _threads())
    if rc != 0:
        raise RuntimeError(f"qxi fill failed ({rc})")
    return out


def weights(dist: str, p: float, seed: int, stream: int, n: int, k: int,
            row0: int = 0, rows: Optional[int] = None) -> np.ndarray:
    """fp32 weight rows [row0, row0+rows) of an n x k matrix (element index r*k + c)."""
    rows = n - row0 if rows is None else rows
    assert 0 <= row0 and row0 + rows <= n
    return fill(dist, p, seed, stream, row0 * k, rows * k, np.float32).reshape(rows, k)


def activations(seed: int, stream: int, count: int, std: float = 1.0,
                outliers: Optional[np.ndarray] = None, outlier_gain: float = 20.0) -> np.ndarray:
    """fp16 N(0, std^2) activations; listed channels are multiplied in fp64 before rounding."""
    v = fill("normal", std, seed, stream, 0, count, np.float64)
    if outliers is not None and len(outliers):
        v = v.copy()
        v[outliers] *= outlier_gain
    return v.astype(np.float16)


def outlier_channels(seed: int, stream: int, k: int, fraction: float = 0.01) -> np.ndarray:
    """round(fraction*k) distinct channels: the smallest keys of one seeded draw."""
    keys = fill("normal", 1.0, seed, stream, 0, k, np.float64)
    cnt = int(round(fraction * k))
    return np.sort(np.argsort(keys, kind="stable")[:cnt])


# ------------------------------------------------------------------ quantizers
@dataclass
class QuantWeight:
    """One group-wise quantized weight matrix, as handed to the packer.

    codes   uint8 [n][k], each < 2**bits
    scales  uint16 [n][k/group] binary16 bits   (uniform only)
    zeros   uint16 [n][k/group] binary16 bits, integer-valued (uniform only)
    codebook uint16 [n][k/group][2**bits] binary16 bits (codebook only);
             for Q4X (kind 2) the matrix's [4][16] codebook
    selectors uint8 [n][k/64], each < 4 (Q4X only)
    """
    n: int
    k: int
    bits: int
    group: int
    kind: int
    codes: np.ndarray
    scales: Optional[np.ndarray] = None
    zeros: Optional[np.ndarray] = None
    codebook: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)
    selectors: Optional[np.ndarray] = None

    def rows(self, r0: int, r1: int) -> "QuantWeight":
        sl = slice(r0, r1)
        per_matrix = self.kind == Q4X  # one codebook for all rows
        return QuantWeight(r1 - r0, self.k, self.bits, self.group, self.kind, self.codes[sl],
                           None if self.scales is None else self.scales[sl],
                           None if self.zeros is None else self.zeros[sl],
                           None if self.codebook is None else (self.codebook if per_matrix else self.codebook[sl]),
                           dict(self.meta), None if self.selectors is None else self.selectors[sl])


def quantize_uniform(w: np.ndarray, bits: int, group: int) -> QuantWeight:
    w = np.ascontiguousarray(w, dtype=np.float32)
    n, k = w.shape
    G = k // group
    codes = np.empty((n, k), np.uint8)
    scales = np.empty((n, G), np.uint16)
    zeros = np.empty((n, G), np.uint16)
    rc = lib().qxi_quantize_uniform(_ptr(w), n, k, bits, group, _ptr(codes), _ptr(scales),
                                    _ptr(zeros), _threads())
    if rc != 0:
        raise ValueError(f"uniform quantization failed ({rc})")
    return QuantWeight(n, k, bits, group, UNIFORM, codes, scales=scales, zeros=zeros)


def quantize_codebook(w: np.ndarray, bits: int, group: int, max_iter: int = 100,
                      keep_raw: bool = False) -> QuantWeight:
    w = np.ascontiguousarray(w, dtype=np.float32)
    n, k = w.shape
    G, E = k // group, 1 << bits
    codes = np.empty((n, k), np.uint8)
    cb = np.empty((n, G, E), np.uint16)
    raw = np.empty((n, G, E), np.float64) if keep_raw else None
    iters = np.empty((n, G), np.int32) if keep_raw else None
    rc = lib().qxi_quantize_codebook(_ptr(w), n, k, bits, group, max_iter, _ptr(codes), _ptr(cb),
                                     _ptr(raw), _ptr(iters), _threads())
    if rc != 0:
        raise ValueError(f"codebook quantization failed ({rc})")
    q = QuantWeight(n, k, bits, group, CODEBOOK, codes, codebook=cb)
    if keep_raw:
        q.meta["raw_centroids"] = raw
        q.meta["iters"] = iters
    return q


def quantize(w: np.ndarray, bits: int, group: int, kind: int) -> QuantWeight:
    if kind == Q4X:
        if bits != 4 or group != 64:
            raise ValueError("Q4X has 4-bit codes in groups of 64")
        from .q4x import quantize_q4x
        return quantize_q4x(w)
    return quantize_uniform(w, bits, group) if kind == UNIFORM else quantize_codebook(w, bits, group)
