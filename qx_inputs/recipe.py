"""Offline recipe: per-matrix format choice and bit allocation by Frobenius error.

The paper keeps both uniform and non-uniform (codebook) group quantization and
chooses between them per matrix from statistics and constraints (Section 2.2),
notes that a matrix better quantized by one kind under the Frobenius norm may not
be better end to end (Section 2.3; its attention-map criterion needs a real model
and is not used here), and that layers may take different bit widths (Section
2.3, last paragraph). On the synthetic weights this tool does the part that
needs no model: for every matrix it measures the relative Frobenius error of each
candidate format on a sample of rows, then allocates formats under a budget of
bits per weight by minimizing the total squared error

    sum_m  ||W_m - W'_m||_F^2   subject to   sum_m bytes_m <= budget.

The allocation is Lagrangian: for a multiplier lam every matrix independently
takes the candidate minimizing err + lam * bytes; lam is bisected to the smallest
value whose allocation fits the budget. An allocation found this way is optimal
among all allocations that use no more bytes than it does (any cheaper-or-equal
allocation with less error would have a smaller Lagrangian). Errors are measured
on the dequantized binary16 weights the kernels use.

CPU only, offline; uses the quantizers of this package. Run as
``python -m qx_inputs.recipe --bpw 4.0``.
"""
from __future__ import annotations

import argparse
import json
from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import CODEBOOK, Q4X, UNIFORM, quantize

# (name, bits, group, kind)
CANDIDATES: Tuple[Tuple[str, int, int, int], ...] = (
    ("U3g128", 3, 128, UNIFORM), ("U3g64", 3, 64, UNIFORM),
    ("U4g128", 4, 128, UNIFORM), ("U4g64", 4, 64, UNIFORM),
    ("CB3g128", 3, 128, CODEBOOK), ("CB4g128", 4, 128, CODEBOOK),
    ("Q4X", 4, 64, Q4X),
)


def bits_per_weight(bits: int, group: int, kind: int) -> float:
    """Code bits plus per-group metadata bits spread over the group."""
    if kind == UNIFORM:
        return bits + 32 / group
    if kind == CODEBOOK:
        return bits + 16 * (1 << bits) / group
    return 4 + 18 / 64  # Q4X: fp16 scale + 2-bit selector per 64 (matrix codebook not counted)


def reconstruct(q) -> np.ndarray:
    """fp16 weights the kernels compute from a quantized matrix, as float64."""
    n, k, g = q.n, q.k, q.group
    j = np.arange(k) // g
    if q.kind == UNIFORM:
        s = q.scales.view(np.float16).astype(np.float64)[:, j]
        z = q.zeros.view(np.float16).astype(np.float64)[:, j]
        return (s * (q.codes - z)).astype(np.float16).astype(np.float64)
    if q.kind == CODEBOOK:
        cb = q.codebook.view(np.float16)
        return cb[np.arange(n)[:, None], j[None, :], q.codes.astype(np.int64)].astype(np.float64)
    s = q.scales.view(np.float16).astype(np.float64)[:, j]
    cb = q.codebook.view(np.float16).astype(np.float64)
    with np.errstate(over="ignore"):
        return (s * cb[q.selectors[:, j], q.codes.astype(np.int64)]).astype(np.float16).astype(np.float64)


@dataclass
class MatrixErrors:
    name: str
    weights: int                 # parameters of the full matrix
    sq_err: Dict[str, float]     # squared Frobenius error per candidate, scaled to the full matrix
    rel_err: Dict[str, float]    # relative Frobenius error on the sample


def measure(name: str, w_sample: np.ndarray, n_full: int,
            candidates: Sequence[Tuple[str, int, int, int]] = CANDIDATES) -> MatrixErrors:
    """Errors of every candidate on a row sample of one matrix (n_full rows in total)."""
    w = np.asarray(w_sample, np.float32)
    ref = w.astype(np.float64)
    norm2 = float((ref * ref).sum())
    scale = n_full / w.shape[0]
    sq, rel = {}, {}
    for cname, bits, group, kind in candidates:
        d = reconstruct(quantize(w, bits, group, kind)) - ref
        e2 = float((d * d).sum())
        sq[cname] = e2 * scale
        rel[cname] = (e2 / norm2) ** 0.5 if norm2 > 0 else 0.0
    return MatrixErrors(name, n_full * w.shape[1], sq, rel)


def _cost(m: MatrixErrors, c: str, candidates) -> float:
    spec = {cn: (b, g, kd) for cn, b, g, kd in candidates}[c]
    return m.weights * bits_per_weight(*spec) / 8.0


def choose(mats: List[MatrixErrors], lam: float, candidates=CANDIDATES) -> Dict[str, str]:
    """Per matrix, the candidate minimizing squared error + lam * bytes (ties: list order)."""
    out = {}
    for m in mats:
        best = min((m.sq_err[c] + lam * _cost(m, c, candidates), i, c)
                   for i, (c, *_rest) in enumerate(candidates))
        out[m.name] = best[2]
    return out


def totals(mats: List[MatrixErrors], alloc: Dict[str, str], candidates=CANDIDATES) -> Tuple[float, float]:
    """(bytes, squared error) of an allocation."""
    b = sum(_cost(m, alloc[m.name], candidates) for m in mats)
    e = sum(m.sq_err[alloc[m.name]] for m in mats)
    return b, e


def allocate(mats: List[MatrixErrors], budget_bytes: float, candidates=CANDIDATES,
             iters: int = 200) -> Dict[str, str]:
    """The Lagrangian allocation with the smallest multiplier that fits the budget.

    Raises ValueError if even the smallest candidate of every matrix exceeds it."""
    hi = 1.0
    while totals(mats, choose(mats, hi, candidates), candidates)[0] > budget_bytes:
        hi *= 4.0
        if hi > 1e30:
            raise ValueError("budget below the smallest format of every matrix")
    lo = 0.0
    if totals(mats, choose(mats, lo, candidates), candidates)[0] <= budget_bytes:
        return choose(mats, lo, candidates)
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if totals(mats, choose(mats, mid, candidates), candidates)[0] <= budget_bytes:
            hi = mid
        else:
            lo = mid
    return choose(mats, hi, candidates)


def decoder_recipe(bpw: float, layers: int = 2, rows: int = 256) -> dict:
    """Recipe for the synthetic 7B decoder's matrices (errors measured on `rows` sampled rows
    of each matrix of the first `layers` layers)."""
    from . import configs
    mats = []
    for layer in range(layers):
        for name in configs.DECODER_MATS:
            spec = configs.c4_matrix(layer, name)
            mats.append(measure(spec.name, spec.weights(0, rows), spec.n))
    total_w = sum(m.weights for m in mats)
    alloc = allocate(mats, bpw * total_w / 8.0)
    b, e = totals(mats, alloc)
    return {"budget_bpw": bpw, "achieved_bpw": 8.0 * b / total_w, "total_sq_err": e,
            "formats": alloc,
            "rel_err": {m.name: round(m.rel_err[alloc[m.name]], 5) for m in mats},
            "candidates_rel_err": {m.name: {c: round(v, 5) for c, v in m.rel_err.items()} for m in mats}}


def main():
    ap = argparse.ArgumentParser(description="per-matrix format allocation by Frobenius error")
    ap.add_argument("--bpw", type=float, default=4.0)
    ap.add_argument("--layers", type=int, default=2)
    ap.add_argument("--rows", type=int, default=256)
    args = ap.parse_args()
    print(json.dumps(decoder_recipe(args.bpw, args.layers, args.rows), indent=1))


if __name__ == "__main__":
    main()
