"""Q4X quantizer: turns fp32 weights into the inputs of the Q4X packer.

The paper describes its Q4X format only in words (Section 3.2, the Q4X item, and
the Figure 3a caption): a histogram per group of 64 weights, 4 histograms learned
to represent all of a matrix's group histograms, each reduced to 16 non-uniform
samples, the 64 samples forming the matrix's codebook; per group a 2-byte scale,
a 2-bit codebook index and 64 4-bit centroid indices. The learning and the
reduction are not specified; this module takes the following reading (every
step deterministic, in fp64):

  1. scale: s16 = the smallest binary16 >= max|w| over the group (1 if the
     group is all zero); u = w / s16 lies in [-1, 1].
  2. histogram: 32 equal bins over [-1, 1] of the group's u, as fractions.
  3. learned histograms: Lloyd's k-means with 4 clusters on the group
     histograms (squared Euclidean distance, evaluated as |c|^2 - 2 h.c; ties
     to the lowest cluster),
     started from the histograms of the groups at ranks (i + 1/2)/4 of the
     mean |u| order, at most 50 iterations; an empty cluster keeps its center.
  4. dimension reduction: each learned histogram, read as a piecewise-uniform
     density on [-1, 1], is reduced to the 16 values of its Lloyd-Max quantizer
     (cells between midpoints of neighbouring values, each value the mean of
     the density over its cell; started at the quantiles (e + 1/2)/16, at most
     100 iterations, an empty cell keeps its value); they are rounded to
     binary16 and sorted ascending: sub-codebook t.
  5. assignment: for each group and each sub-codebook t, every weight takes the
     index of its nearest dequantized level fp16(s16 * CB[t][e]) (ties to the
     lowest index); the group's selector is the t with the least squared error
     (ties to the lowest t).
"""
from __future__ import annotations

import numpy as np

from . import Q4X, QuantWeight, _ptr, _threads, double_to_half_bits, lib

GROUP, SUBBOOKS, ENTRIES, BINS = 64, 4, 16, 32


def _scales(wg: np.ndarray) -> np.ndarray:
    amax = np.max(np.abs(wg), axis=1)
    s = double_to_half_bits(amax, 1)  # toward +inf: |w| <= s16
    s[amax == 0] = 0x3C00
    return s


def _histograms(w32: np.ndarray, s16: np.ndarray) -> np.ndarray:
    """Step 2 (native): [groups][32] bin fractions of w / s16."""
    ng = s16.size
    h = np.empty((ng, BINS))
    lib().qxi_q4x_histograms(_ptr(w32), ng, _ptr(s16), _ptr(h), _threads())
    return h


def _nearest_center(h: np.ndarray, centers: np.ndarray) -> np.ndarray:
    # squared distance up to the per-row constant |h|^2: |c|^2 - 2 h.c
    d = (centers * centers).sum(axis=1)[None, :] - 2.0 * (h @ centers.T)
    return np.argmin(d, axis=1)  # first minimum: ties go to the lowest cluster


def learn_histograms(h: np.ndarray, mean_abs_u: np.ndarray, max_iter: int = 50):
    """Step 3: (centers [4][32], assignment, iterations run)."""
    order = np.argsort(mean_abs_u, kind="stable")
    picks = order[((np.arange(SUBBOOKS) + 0.5) / SUBBOOKS * len(order)).astype(np.int64)]
    centers = h[picks].copy()
    assign = _nearest_center(h, centers)
    it = 0
    for it in range(1, max_iter + 1):
        onehot = (assign[:, None] == np.arange(SUBBOOKS)[None, :]).astype(np.float64)
        count = onehot.sum(axis=0)
        sums = onehot.T @ h
        for t in range(SUBBOOKS):
            if count[t]:
                centers[t] = sums[t] / count[t]
        new = _nearest_center(h, centers)
        if np.array_equal(new, assign):
            break
        assign = new
    return centers, assign, it


def _quantiles(pmf: np.ndarray, edges: np.ndarray) -> np.ndarray:
    cdf = np.concatenate([[0.0], np.cumsum(pmf)])
    cdf /= cdf[-1]
    out = np.empty(ENTRIES)
    for e in range(ENTRIES):
        p = (e + 0.5) / ENTRIES
        i = int(np.searchsorted(cdf, p, side="right")) - 1  # cdf[i] <= p < cdf[i+1]
        i = min(max(i, 0), BINS - 1)
        width = cdf[i + 1] - cdf[i]
        frac = 0.0 if width == 0 else (p - cdf[i]) / width
        out[e] = edges[i] + frac * (edges[i + 1] - edges[i])
    return out


def _cell_moments(pmf: np.ndarray, edges: np.ndarray, lo: float, hi: float):
    """Mass and first moment of the piecewise-uniform density over [lo, hi]."""
    a = np.clip(edges[:-1], lo, hi)
    b = np.clip(edges[1:], lo, hi)
    dens = pmf / (edges[1:] - edges[:-1])
    return float((dens * (b - a)).sum()), float((dens * (b * b - a * a) / 2.0).sum())


def reduce_histogram(pmf: np.ndarray, max_iter: int = 100) -> np.ndarray:
    """Step 4: the 16 Lloyd-Max values (fp64, ascending) of one learned histogram."""
    edges = np.linspace(-1.0, 1.0, BINS + 1)
    c = _quantiles(pmf, edges)
    for _ in range(max_iter):
        bounds = np.concatenate([[-1.0], (c[:-1] + c[1:]) / 2.0, [1.0]])
        new = c.copy()
        for e in range(ENTRIES):
            mass, moment = _cell_moments(pmf, edges, bounds[e], bounds[e + 1])
            if mass > 0:
                new[e] = moment / mass
        if np.max(np.abs(new - c)) < 1e-12:
            c = new
            break
        c = new
    return c


def assign_codes(w32: np.ndarray, s16: np.ndarray, codebook: np.ndarray):
    """Step 5 (native): (codes [groups][64], selectors [groups])."""
    ng = s16.size
    codes = np.empty((ng, GROUP), np.uint8)
    sel = np.empty(ng, np.uint8)
    cb = np.ascontiguousarray(codebook, np.uint16)
    lib().qxi_q4x_assign(_ptr(w32), ng, _ptr(s16), _ptr(cb), _ptr(codes), _ptr(sel), _threads())
    return codes, sel


def assign_codes_numpy(wg: np.ndarray, s16: np.ndarray, codebook: np.ndarray, chunk: int = 4096):
    """Step 5 in numpy (fp64 brute force), the check of :func:`assign_codes`."""
    s = s16.view(np.float16).astype(np.float64)
    cb = codebook.view(np.float16).astype(np.float64)
    ng = wg.shape[0]
    codes = np.empty(wg.shape, np.uint8)
    sel = np.empty(ng, np.uint8)
    for a in range(0, ng, chunk):
        w = wg[a:a + chunk]
        best_err = np.full(w.shape[0], np.inf)
        for t in range(SUBBOOKS):
            levels = (s[a:a + chunk, None] * cb[t][None, :]).astype(np.float16).astype(np.float64)
            d = np.abs(w[:, :, None] - levels[:, None, :])
            q = np.argmin(d, axis=2)  # ties to the lowest index
            err = (np.take_along_axis(d, q[:, :, None], axis=2)[:, :, 0] ** 2).sum(axis=1)
            better = err < best_err  # ties keep the lower selector
            best_err[better] = err[better]
            sel[a:a + chunk][better] = t
            codes[a:a + chunk][better] = q[better]
    return codes, sel


def quantize_q4x(w: np.ndarray, max_iter: int = 50) -> QuantWeight:
    """Q4X quantization of fp32 weights [n][k] (k a multiple of 128).

    Returns a QuantWeight with kind Q4X, bits 4, group 64: codes [n][k], scales
    [n][k/64] (binary16 bits), selectors [n][k/64] (uint8 < 4) and codebook
    [4][16] (binary16 bits, the matrix's 64 centroids)."""
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    if k % 128:
        raise ValueError("k must be a multiple of 128")
    G = k // GROUP
    w32 = np.ascontiguousarray(w)
    wg = w32.reshape(n * G, GROUP)
    s16 = np.ascontiguousarray(_scales(wg))
    h = _histograms(w32, s16)
    mean_abs = np.mean(np.abs(wg.astype(np.float64)), axis=1) / s16.view(np.float16).astype(np.float64)
    centers, _, iters = learn_histograms(h, mean_abs, max_iter)
    samples = np.stack([reduce_histogram(centers[t]) for t in range(SUBBOOKS)])
    cb = double_to_half_bits(samples, 0)
    cb = np.stack([np.sort(cb[t].view(np.float16), kind="stable").view(np.uint16) for t in range(SUBBOOKS)])
    codes, sel = assign_codes(w32, s16, cb)
    q = QuantWeight(n, k, 4, GROUP, Q4X, codes.reshape(n, k), scales=s16.reshape(n, G), codebook=cb,
                    selectors=sel.reshape(n, G))
    q.meta["kmeans_iters"] = iters
    q.meta["learned_histograms"] = centers
    return q
