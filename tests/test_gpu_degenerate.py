"""Uniform groups whose weights are all zero, through the GEMV and the small-batch GEMM.

The uniform quantizer stores such a group with s = 1, z = 0 and every code 0
(the levels s(q - z) of Section 2.2 are then all zero). The GEMV kernels fold
the zero point out of their inner loop, so the group's sum of (M + q)x and the
staged sum of M x must cancel exactly for it: they are formed by the same
instructions in the same order. These tests mix quantizer-made all-zero groups
and all-zero rows into small-weight (N(0, 0.002)) and heavy-tailed (Student-t,
std 0.02) matrices, multiply them with activations that carry 1 % outlier
channels x20, and require every output vector within 2e-3 of the oracle and the
all-zero rows to come out exactly 0.
"""
import numpy as np
import pytest

import oracle
import qx_inputs as qi
from helpers import TOL, to_dev

pytestmark = pytest.mark.gpu

FORMATS = [(b, g) for b in (3, 4) for g in (32, 64, 128)]
DISTS = [("normal", 0.002), ("t4", 0.02)]
# rows of 32 chunks (in-wave reduction), 86 chunks (row kernel), 96 chunks (k tiles), and a
# matrix with more rows than columns (m = 3, 4 then run on the matrix cores)
SHAPES = [(300, 4096), (200, 11008), (40, 12288), (2048, 1024)]


def _weights_with_zero_groups(dist, p, n, k, group, seed):
    w = qi.weights(dist, p, seed, 0, n, k).copy()
    rng = np.random.default_rng(seed)
    w[::7] = 0.0                                       # whole rows
    zero = rng.random((n, k // group)) < 0.2           # ~20 % of the other groups
    w.reshape(n, k // group, group)[zero] = 0.0
    return w


def _x(k, seed, m=None):
    rows = []
    for r in range(1 if m is None else m):
        out = qi.outlier_channels(seed + r, 2, k, 0.01)
        rows.append(qi.activations(seed + r, 1, k, outliers=out))
    return rows[0] if m is None else np.stack(rows)


@pytest.mark.parametrize("fmt", FORMATS, ids=lambda f: f"u{f[0]}g{f[1]}")
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: d[0])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_zero_groups_and_rows(gpu, fmt, dist, shape):
    qx = gpu
    bits, g = fmt
    n, k = shape
    seed = 17 * n + k + 3 * bits + g
    print(f"zero groups u{bits}g{g} {dist[0]} {shape}", flush=True)
    w = _weights_with_zero_groups(dist[0], dist[1], n, k, g, seed)
    q = qi.quantize(w, bits, g, qi.UNIFORM)
    zg = np.all(w.reshape(n, k // g, g) == 0, axis=2)
    assert zg.any()
    assert np.all(q.scales[zg] == 0x3C00) and np.all(q.zeros[zg] == 0)  # s = 1, z = 0
    assert np.all(q.codes.reshape(n, k // g, g)[zg] == 0)
    zero_rows = np.all(w == 0, axis=1)
    w16 = oracle.dequant(q.codes, g, q.kind, q.scales, q.zeros, q.codebook)
    pw = qx.PackedWeight.from_quant(q)

    x = _x(k, seed)
    y = pw.gemv(to_dev(x)).cpu().numpy()
    err = oracle.normwise_rel_err(y, oracle.gemv(w16, x))
    print(f"  gemv normwise rel err {err:.3e}")
    assert err <= TOL, err
    assert np.all(y[zero_rows] == 0)

    for m in (2, 3, 4):
        X = _x(k, seed + 100, m)
        Y = pw.gemm(to_dev(X)).cpu().numpy()
        ref = oracle.gemm(X, w16)
        errs = [oracle.normwise_rel_err(Y[r], ref[r]) for r in range(m)]
        print(f"  gemm m={m} max normwise rel err {max(errs):.3e}")
        assert max(errs) <= TOL, (m, errs)
        assert np.all(Y[:, zero_rows] == 0)
