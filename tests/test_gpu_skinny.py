"""Parity of the small-batch matrix-core GEMM (qx_gemm at 2 <= m <= 64) with the oracle.

That kernel keeps the GEMV's one-chunk-per-lane loads and multiplies on the
matrix cores: a block's waves split each row's chunks 4 per wave and item (up
to 4 items per lane, up to 8 waves) on 16, 32, 48 or 96 weight rows per block
(one, two, three or six row fragments per wave), each wave stages the m activation rows of
its chunks in LDS, and the m rows fill 16-row tiles taken in turn (more than one
only on rows of at most 32 chunks). Tall matrices with rows of 29-32 chunks at m <= 16
take a pipelined form instead (one block per compute unit walking 16-row groups with
two in flight). The cases below take
each of those launch shapes at an m and shape that qx_gemm routes to it, with
ragged rows, chunk slots past the end of a row, waves without a last item and
padded activation rows, in all thirteen formats (where a format is routed
elsewhere the case checks that path). Every output row must be within the
normwise bound of the oracle; a one-hot activation row must reproduce a column
of W' exactly (the products are exact and the matrix cores add zeros), and
repeated runs must be bitwise identical.
"""
import numpy as np
import pytest

import oracle
from oracle import q4x
import qx_inputs as qi
from qx_inputs import q4x as qq
from helpers import TOL, activations, random_quant, to_dev

pytestmark = pytest.mark.gpu

FORMATS = [(b, kind, g) for b in (3, 4) for kind in (0, 1) for g in (32, 64, 128)] + [(4, 2, 64)]

# (m, n, k): chunks per row C = k / 128 give 1-4 items per lane (C <= 32, 64, 96, 128)
# and 1-8 waves; 8192 rows or more take 3 (one item) or 2 (two items) row fragments
CASES = [
    (2, 40, 384),       # C = 3: one wave, lane group 3 past the row
    (5, 37, 1152),      # C = 9: 3 waves, the last with one valid lane group
    (16, 130, 4096),    # C = 32: 8 waves, a full activation tile
    (3, 9, 8192),       # C = 64: 2 items, 8 waves; n < 16
    (12, 100, 11008),   # C = 86: 3 items, 8 waves, two waves without a third
    (4, 8200, 4096),    # three row fragments per wave, last block ragged (40 of 48 rows)
    (16, 8200, 4096),   # the same at a full activation tile
    (7, 8193, 5120),    # C = 40: two row fragments per wave and 2 items; one row in the last block
    (6, 60, 16384),     # C = 128: 4 items, 8 waves
    (2, 37, 11008),     # m = 2 on 3 items (uniform and codebook codes here since the one-item look-ahead)
    (2, 20, 16384),     # m = 2 on 4 items: codebooks here, uniform codes GEMV-style
    (24, 130, 4096),    # two activation tiles, the second of 8 rows
    (33, 8200, 4096),   # three tiles (the last of one row), three row fragments per wave
    (64, 40, 384),      # four full tiles, one wave
    (47, 8193, 1152),   # three tiles, three fragments, one row in the last block
    (56, 8200, 4096),   # four tiles (the last of 8 rows), three fragments per wave
    (9, 16400, 1024),   # six row fragments per wave (16384 rows or more), last block of 80 rows
    (2, 8190, 4096),    # pipelined form: two 16-row groups per compute unit, the last of 14 rows
    (16, 16390, 3840),  # pipelined, C = 30 (lane groups past the row), 4-5 groups per block, last of 6 rows
    (7, 22001, 4096),   # pipelined, 5-6 groups per block (both tails), the last of one row
    (3, 20, 22016),     # C = 172: past the kernel's rows, routed elsewhere
    (4, 33, 32768),     # C = 256: routed elsewhere
]


def _fmt_id(f):
    return f"b{f[0]}{'ucq'[f[1]]}g{f[2]}"


def _quant(n, k, fmt, seed):
    bits, kind, g = fmt
    if kind == 2:
        rng = np.random.default_rng(seed)
        G = k // 64
        s = np.float16(rng.uniform(0.25, 2.0, (n, G)) * rng.choice([-1.0, 1.0], (n, G), p=[0.1, 0.9]))
        cb = np.sort(rng.standard_normal((4, 16)) * 0.05, axis=1).astype(np.float16).view(np.uint16)
        return qi.QuantWeight(n, k, 4, 64, qq.Q4X, rng.integers(0, 16, (n, k), dtype=np.uint8),
                              scales=s.view(np.uint16), codebook=cb,
                              selectors=rng.integers(0, 4, (n, G), dtype=np.uint8))
    return random_quant(n, k, bits, g, kind, seed=seed)


def _w16(q, rows=None):
    """W' (fp16 values) of all rows, or of the given rows only."""
    def sel(a):
        return a if a is None or rows is None else a[rows]
    if q.kind == 2:  # the codebook is per matrix
        return q4x.dequant(sel(q.codes), sel(q.scales), sel(q.selectors), q.codebook)
    return oracle.dequant(sel(q.codes), q.group, q.kind, sel(q.scales), sel(q.zeros), sel(q.codebook))


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"m{c[0]}_{c[1]}x{c[2]}")
def test_skinny_matches_oracle(gpu, fmt, case):
    qx = gpu
    m, n, k = case
    print(f"skinny {_fmt_id(fmt)} m={m} {n}x{k}", flush=True)
    q = _quant(n, k, fmt, seed=n + k + m)
    X = activations(k, seed=m + 7, m=m)
    pw = qx.PackedWeight.from_quant(q)
    Y = pw.gemm(to_dev(X)).cpu().numpy()
    rows = np.arange(n) if n <= 1024 else np.sort(np.random.default_rng(m).choice(n, 1024, replace=False))
    rows = np.union1d(rows, [n - 1])  # the ragged last block
    ref = oracle.gemm(X, _w16(q, rows))
    for r in range(m):
        err = oracle.normwise_rel_err(Y[r][rows], ref[r])
        assert err <= TOL, (r, err)
    Y2 = pw.gemm(to_dev(X)).cpu().numpy()
    assert np.array_equal(Y.view(np.uint16), Y2.view(np.uint16))  # deterministic


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("m,n,k", [(4, 8200, 11008), (6, 4000, 11008), (16, 8200, 4096), (40, 4096, 4096),
                                   (5, 16400, 4096)],
                         ids=["m4_8200x11008", "m6_4000x11008", "m16_8200x4096", "m40_4096x4096", "m5_16400x4096"])
def test_skinny_one_hot_rows_are_columns(gpu, fmt, m, n, k):
    """Activation row r one-hot at position j_r: row r of Y equals column j_r of W' in
    value (a sum that starts at +0 turns -0 weights into +0), on shapes with 3 items per
    lane and a ragged last item (16-row blocks), with 48-row blocks at m = 16, with three
    activation tiles at m = 40, and in the pipelined form (16400 rows)."""
    qx = gpu
    q = _quant(n, k, fmt, seed=m)
    cols = np.random.default_rng(m + 1).choice(k, m, replace=False)
    X = np.zeros((m, k), np.float16)
    X[np.arange(m), cols] = 1.0
    Y = qx.PackedWeight.from_quant(q).gemm(to_dev(X)).cpu().numpy()
    ref = _w16(q)[:, cols].T
    assert np.array_equal(Y.astype(np.float32), ref.astype(np.float32))


@pytest.mark.parametrize("m", [2, 6, 8, 13, 16, 40])
def test_skinny_rows_equal_gemv(gpu, m):
    """Each row of the product against the batch-1 GEMV of the same row (two different
    fp32 summation orders of the same products)."""
    qx = gpu
    q = random_quant(1000, 4096, 3, 64, 0, seed=m)
    pw = qx.PackedWeight.from_quant(q)
    X = activations(4096, seed=m + 1, m=m)
    Y = pw.gemm(to_dev(X)).cpu().numpy()
    for r in range(m):
        y = pw.gemv(to_dev(X[r])).cpu().numpy()
        assert oracle.normwise_rel_err(Y[r], y.astype(np.float64)) <= 2 * TOL, r

