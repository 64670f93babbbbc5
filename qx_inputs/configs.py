"""The five synthetic workloads, by seed, stream, shape and distribution.

Shapes are those of a 7B decoder (hidden 4096, MLP 11008, 32 layers, q/k/v/o
4096x4096, gate/up 11008x4096, down 4096x11008); weight rows are output
features and groups run along the reduction axis. Distributions follow the
paper's observation that attention weights are narrow and peaked while MLP
weights are wider (Section 2.1), and that activations carry outlier channels
(Section 2.4). Every matrix is a (seed, stream) pair of the Philox generator,
so any row can be regenerated alone.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

from . import (CODEBOOK, Q4X, UNIFORM, QuantWeight, activations, fill, outlier_channels, quantize,
               weights)

HIDDEN, MLP, LAYERS = 4096, 11008, 32
LAPLACE_B = 0.008   # narrow, peaked attention weights
T4_STD = 0.02       # heavy-tailed MLP weights (Student-t, 4 degrees of freedom)


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    n: int
    k: int
    dist: str
    p: float
    seed: int
    stream: int
    bits: int
    group: int
    kind: int

    def weights(self, row0: int = 0, rows: Optional[int] = None) -> np.ndarray:
        return weights(self.dist, self.p, self.seed, self.stream, self.n, self.k, row0, rows)

    def quantized(self, row0: int = 0, rows: Optional[int] = None) -> QuantWeight:
        """The quantized rows [row0, row0 + rows), from the disk cache when present."""
        from . import cache
        q = cache.load(self, row0, rows)
        if q is None:
            q = quantize(self.weights(row0, rows), self.bits, self.group, self.kind)
            cache.store(self, row0, rows, q)
        q.meta["spec"] = self
        q.meta["row0"] = row0
        return q

    @property
    def packed_bytes(self) -> int:
        """Code bytes plus per-group table bytes (the bits-per-weight footprint); for Q4X
        also the per-row selector words, the alignment padding and the 128-byte codebook."""
        G = self.k // self.group
        if self.kind == Q4X:
            sel_words = self.n * ((G + 15) // 16) * 4
            return (self.n * self.k // 2 + self.n * G * 2 + sel_words + 15) // 16 * 16 + 128
        meta = 4 if self.kind == UNIFORM else 2 * (1 << self.bits)
        return self.n * self.k * self.bits // 8 + self.n * G * meta


def c1():
    """4096x4096, N(0, 0.02) weights, 4-bit uniform, group 128; x ~ N(0,1)."""
    w = MatrixSpec("c1", HIDDEN, HIDDEN, "normal", 0.02, 0, 0, 4, 128, UNIFORM)
    return w, activations(0, 1, HIDDEN)


def c2():
    """11008x4096 Student-t(4) std 0.02, 3-bit uniform, group 64; x ~ N(0,1) with 1% of
    channels x20."""
    w = MatrixSpec("c2", MLP, HIDDEN, "t4", T4_STD, 1, 0, 3, 64, UNIFORM)
    out = outlier_channels(1, 2, HIDDEN, 0.01)
    return w, activations(1, 1, HIDDEN, outliers=out)


def c3():
    """4096x4096 Laplace(0, 0.008), 3-bit per-group codebook (8 fp16 entries), group 128."""
    w = MatrixSpec("c3", HIDDEN, HIDDEN, "laplace", LAPLACE_B, 2, 0, 3, 128, CODEBOOK)
    return w, activations(2, 1, HIDDEN)


DECODER_MATS = ("q", "k", "v", "o", "gate", "up", "down")
# activation t of layer l: 0 = attention input (q, k, v), 1 = o input, 2 = MLP input (gate, up),
# 3 = down input
DECODER_X = {"q": 0, "k": 0, "v": 0, "o": 1, "gate": 2, "up": 2, "down": 3}


def c4_matrix(layer: int, name: str) -> MatrixSpec:
    """One weight of the 32-layer decoder: attention 3-bit codebook g128 (Laplace), MLP 4-bit
    uniform g128 (Student-t(4))."""
    j = DECODER_MATS.index(name)
    seed, stream = 3, 7 * layer + j
    if name in ("q", "k", "v", "o"):
        return MatrixSpec(f"L{layer}.{name}", HIDDEN, HIDDEN, "laplace", LAPLACE_B, seed, stream,
                          3, 128, CODEBOOK)
    if name in ("gate", "up"):
        return MatrixSpec(f"L{layer}.{name}", MLP, HIDDEN, "t4", T4_STD, seed, stream, 4, 128,
                          UNIFORM)
    return MatrixSpec(f"L{layer}.down", HIDDEN, MLP, "t4", T4_STD, seed, stream, 4, 128, UNIFORM)


def c4_activation(layer: int, t: int) -> np.ndarray:
    return activations(3, 1000 + 4 * layer + t, MLP if t == 3 else HIDDEN)


def c4_batch_activations(layer: int, t: int, m: int) -> np.ndarray:
    """[m][k] activations of m sequences decoded together; row 0 is c4_activation(layer, t)."""
    count = MLP if t == 3 else HIDDEN
    return np.stack([activations(3, 1000 + 4 * layer + t + 4096 * r, count) for r in range(m)])


def c4_plan(layers: int = LAYERS) -> List[tuple]:
    """(spec, activation index) for every GEMV of one decode step, in launch order."""
    return [(c4_matrix(l, m), (l, DECODER_X[m])) for l in range(layers) for m in DECODER_MATS]


C5_M = (16, 64, 512)


def c5_matrix(name: str) -> MatrixSpec:
    """Prefill MLP weights: gate/up 11008x4096, down 4096x11008, Student-t(4), 3-bit uniform g64."""
    j = ("gate", "up", "down").index(name)
    n, k = (MLP, HIDDEN) if name != "down" else (HIDDEN, MLP)
    return MatrixSpec(f"c5.{name}", n, k, "t4", T4_STD, 4, j, 3, 64, UNIFORM)


def c5_activations(m: int) -> tuple:
    """(X_in [m][4096] shared by gate and up, X_down [m][11008]) fp16 N(0,1)."""
    xin = fill("normal", 1.0, 4, 10_000 + m, 0, m * HIDDEN).astype(np.float16).reshape(m, HIDDEN)
    xdn = fill("normal", 1.0, 4, 20_000 + m, 0, m * MLP).astype(np.float16).reshape(m, MLP)
    return xin, xdn


def q4x_matrix(name: str) -> MatrixSpec:
    """The paper's Q4X format (4-bit indices into a per-matrix 4 x 16 codebook, groups of 64)
    on MLP-shaped weights: gate 11008x4096 and down 4096x11008, Student-t(4) std 0.02."""
    j = ("gate", "down").index(name)
    n, k = (MLP, HIDDEN) if name == "gate" else (HIDDEN, MLP)
    return MatrixSpec(f"q4x.{name}", n, k, "t4", T4_STD, 5, j, 4, 64, Q4X)


def q4x_activation(name: str) -> np.ndarray:
    return activations(5, 100 + ("gate", "down").index(name), HIDDEN if name == "gate" else MLP)
