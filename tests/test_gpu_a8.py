"""Parity of the 8-bit-activation GEMV (qx_gemv_a8, through the C ABI) with the
oracle: per-token symmetric RTN of x to int8 (Section 2.4; the W3A8 rows of
Table 1), integer products with the uniform codes, y = s_x * sum_j s_j *
sum (q - z) * xq. The int8 codes are decided in fp32 on both sides, the sums are
exact integers, so the only differences are the fp32 scaling and the fp16 output
rounding: the normwise bound of the other GEMVs applies with room to spare."""
import numpy as np
import pytest

import oracle
from oracle import a8
import qx_inputs as qi
from helpers import TOL, activations, random_quant, realistic_quant, to_dev

pytestmark = pytest.mark.gpu

FORMATS = [(b, g) for b in (3, 4) for g in (32, 64, 128)]
SHAPES = [(1, 128), (3, 384), (37, 256), (9, 1152), (5, 11008), (130, 4096), (260, 1024),
          (19, 8192), (1001, 11008), (4096, 4096)]


@pytest.mark.parametrize("fmt", FORMATS, ids=lambda f: f"b{f[0]}g{f[1]}")
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_gemv_a8_matches_oracle(gpu, fmt, shape):
    qx = gpu
    bits, g = fmt
    n, k = shape
    print(f"a8 gemv {fmt} {shape}", flush=True)
    q = realistic_quant(n, k, bits, g, 0, seed=n + k + bits)
    x = activations(k, seed=k + g)
    y = qx.PackedWeight.from_quant(q).gemv_a8(to_dev(x)).cpu().numpy()
    err = oracle.normwise_rel_err(y, a8.gemv_a8(q.codes, g, q.scales, q.zeros, x))
    assert err <= TOL, err


def test_gemv_a8_outlier_activations_and_c2(gpu):
    """c2's activations have 1 % of channels x20, so the int8 step is coarse for the rest:
    still the integer path's own definition, matched within the bound."""
    qx = gpu
    from qx_inputs import configs
    spec, x = configs.c2()
    q = spec.quantized()
    y = qx.PackedWeight.from_quant(q).gemv_a8(to_dev(x)).cpu().numpy()
    err = oracle.normwise_rel_err(y, a8.gemv_a8(q.codes, spec.group, q.scales, q.zeros, x))
    assert err <= TOL, err


@pytest.mark.parametrize("k", [128, 4096, 11008])
def test_gemv_a8_zero_and_determinism(gpu, k):
    qx = gpu
    q = realistic_quant(70, k, 4, 128, 0, seed=k)
    pw = qx.PackedWeight.from_quant(q)
    assert np.all(pw.gemv_a8(to_dev(np.zeros(k, np.float16))).cpu().numpy() == 0)
    xd = to_dev(activations(k, seed=3))
    a = pw.gemv_a8(xd).cpu().numpy()
    b = pw.gemv_a8(xd).cpu().numpy()
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


def test_gemv_a8_single_nonzero_activation(gpu):
    """x = c * e_j: xq is 127 at j, so y = s_x * 127 * s * (q - z) for the column's group."""
    qx = gpu
    n, k = 64, 1024
    q = realistic_quant(n, k, 3, 64, 0, seed=9)
    pw = qx.PackedWeight.from_quant(q)
    for j in (0, 500, k - 1):
        x = np.zeros(k, np.float16)
        x[j] = -0.75
        y = pw.gemv_a8(to_dev(x)).cpu().numpy()
        ref = a8.gemv_a8(q.codes, 64, q.scales, q.zeros, x)
        assert oracle.normwise_rel_err(y, ref) <= 2.0**-10, j


# ------------------------------------------------------------ many rows: qx_gemm_a8
def _x_rows(m, k, seed):
    X = activations(k, seed=seed, m=m)
    if m > 2:
        X[1] = 0                                    # an all-zero token: xq = 0, s_x = 0
        X[2, (seed * 7) % k] = np.float16(65504.0)  # one huge value: every other code rounds to ~0
    return X


@pytest.mark.parametrize("m,k", [(1, 128), (5, 384), (37, 4096), (130, 11008), (7, 1 << 14)])
def test_quantize_a8_rows_bit_exact(gpu, m, k):
    """qx_quantize_a8 takes each row's integer decision exactly as the oracle: int8 codes
    and the fp32 scale bit for bit (zero row and single huge value included)."""
    qx = gpu
    X = _x_rows(m, k, seed=m + k)
    Xq, sx = qx.quantize_a8(to_dev(X))
    Xq, sx = Xq.cpu().numpy(), sx.cpu().numpy()
    for r in range(m):
        q, s = a8.quantize_activation(X[r])
        assert np.array_equal(Xq[r], q), r
        assert np.float32(sx[r]).view(np.uint32) == np.float32(s).view(np.uint32), r


GEMM_A8 = [(1, 40, 1152), (3, 100, 384), (16, 130, 4096), (17, 64, 11008), (33, 300, 1024),
           (64, 257, 4096), (65, 64, 2048), (512, 200, 4096), (3, 9, 1 << 18), (256, 4096, 512),
           (130, 2000, 1024)]


@pytest.mark.parametrize("fmt", FORMATS, ids=lambda f: f"b{f[0]}g{f[1]}")
@pytest.mark.parametrize("m,n,k", GEMM_A8, ids=lambda v: str(v))
def test_gemm_a8_matches_oracle(gpu, fmt, m, n, k):
    """Every row of qx_gemm_a8 against the oracle's per-token A8 GEMV of that row."""
    qx = gpu
    bits, g = fmt
    print(f"a8 gemm {fmt} m={m} {n}x{k}", flush=True)
    q = realistic_quant(n, k, bits, g, 0, seed=n + k + m + bits)
    X = _x_rows(m, k, seed=k + g + m)
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = qx.PackedWeight.from_quant(q).gemm_a8(Xq, sx).cpu().numpy()
    for r in range(m):
        ref = a8.gemv_a8(q.codes, g, q.scales, q.zeros, X[r])
        if not np.any(ref):
            assert not np.any(Y[r].astype(np.float32)), r
            continue
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, (r, oracle.normwise_rel_err(Y[r], ref))


@pytest.mark.parametrize("fmt", [(3, 64), (4, 128), (3, 32)], ids=lambda f: f"b{f[0]}g{f[1]}")
@pytest.mark.parametrize("m,n", [(16, 300), (64, 300), (200, 4096), (512, 4096)], ids=lambda v: str(v))
def test_gemm_a8_long_rows(gpu, fmt, m, n):
    """Rows of more than 64 chunks (k = 11008), where the k split runs over 8 waves, at every
    tile shape by m; sampled rows against the oracle's per-token A8 GEMV."""
    qx = gpu
    bits, g = fmt
    k = 11008
    print(f"a8 gemm long rows {fmt} m={m} n={n}", flush=True)
    q = random_quant(n, k, bits, g, 0, seed=m + n + g)
    X = _x_rows(m, k, seed=m + g)
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = qx.PackedWeight.from_quant(q).gemm_a8(Xq, sx).cpu().numpy()
    for r in sorted(set(range(0, m, max(1, m // 6))) | {1, m - 1}):
        ref = a8.gemv_a8(q.codes, g, q.scales, q.zeros, X[r])
        if not np.any(ref):  # the all-zero token
            assert not np.any(Y[r].astype(np.float32)), r
            continue
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, r


@pytest.mark.parametrize("bits,g", [(3, 128), (4, 32)])
def test_gemm_a8_integer_results_are_exact(gpu, bits, g):
    """Scales 1, activations integers with one entry 127 per row (so inv = 1 and s_x = 1
    exactly; that column's codes equal the zero point): every output is the integer sum
    of (q - z) * x, small enough to be exact in binary16, bit for bit."""
    qx = gpu
    n, k, m = 80, 1024, 48
    rng = np.random.default_rng(bits * g)
    G = k // g
    codes = rng.integers(0, 2 ** bits, (n, k), dtype=np.uint8)
    zeros = rng.integers(0, 2 ** bits, (n, G)).astype(np.float16).view(np.uint16)
    scales = np.ones((n, G), np.float16).view(np.uint16)
    q = qi.QuantWeight(n, k, bits, g, 0, codes, scales=scales, zeros=zeros)
    codes[:, 5] = zeros.view(np.float16)[:, 5 // g].astype(np.uint8)  # q - z = 0 where x = 127
    X = rng.integers(-1, 2, (m, k)).astype(np.float16)
    X[:, 5] = 127
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = qx.PackedWeight.from_quant(q).gemm_a8(Xq, sx).cpu().numpy()
    d = codes.astype(np.int64) - np.repeat(zeros.view(np.float16).astype(np.int64), g, axis=1)
    ref = X.astype(np.int64) @ d.T
    assert np.abs(ref).max() < 2048
    assert np.array_equal(Y.astype(np.float32), ref.astype(np.float32))


def test_gemm_a8_rows_equal_gemv_a8_within_tolerance_and_repeat_bitwise(gpu):
    qx = gpu
    q = realistic_quant(500, 4096, 3, 128, 0, seed=9)
    pw = qx.PackedWeight.from_quant(q)
    X = activations(4096, seed=4, m=6)
    Xd = to_dev(X)
    Xq, sx = qx.quantize_a8(Xd)
    Y1 = pw.gemm_a8(Xq, sx).cpu().numpy()
    Y2 = pw.gemm_a8(Xq, sx).cpu().numpy()
    assert np.array_equal(Y1.view(np.uint16), Y2.view(np.uint16))
    for r in range(6):
        y = pw.gemv_a8(Xd[r].contiguous()).cpu().numpy()
        assert oracle.normwise_rel_err(Y1[r], y.astype(np.float64)) <= TOL


@pytest.mark.parametrize("fmt", FORMATS, ids=lambda f: f"b{f[0]}g{f[1]}")
@pytest.mark.parametrize("n,k", [(300, 4096), (70, 8192), (130, 11008), (37, 1152), (9, 1 << 14)])
def test_gemm_a8_one_row_is_the_a8_gemv(gpu, fmt, n, k):
    """m = 1 with k <= 88 chunks runs the A8 GEMV on the pre-quantized row: qx_gemv_a8's bits
    (it quantizes the same fp16 row to the same codes); longer k runs the matrix cores and is
    held to the oracle."""
    qx = gpu
    bits, g = fmt
    q = random_quant(n, k, bits, g, 0, seed=n + k + g)
    pw = qx.PackedWeight.from_quant(q)
    x = activations(k, seed=k + bits)
    xd = to_dev(x)
    Xq, sx = qx.quantize_a8(xd[None, :].contiguous())
    a = pw.gemm_a8(Xq, sx).cpu().numpy()[0]
    if k <= 88 * 128:
        b = pw.gemv_a8(xd).cpu().numpy()
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    else:
        assert oracle.normwise_rel_err(a, a8.gemv_a8(q.codes, g, q.scales, q.zeros, x)) <= TOL


@pytest.mark.parametrize("fmt", FORMATS, ids=lambda f: f"b{f[0]}g{f[1]}")
@pytest.mark.parametrize("m", [2, 3, 4])
@pytest.mark.parametrize("n,k", [(4096, 4096), (300, 11008), (37, 1152), (9, 1 << 16)])
def test_gemm_a8_small_batch(gpu, fmt, m, n, k):
    """2 <= m <= 4 pre-quantized rows run the small-batch A8 kernel (each code decoded once
    for all rows); every row against the oracle's A8 GEMV of that row."""
    qx = gpu
    bits, g = fmt
    q = random_quant(n, k, bits, g, 0, seed=n + k + m)
    X = _x_rows(m, k, seed=k + m)
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = qx.PackedWeight.from_quant(q).gemm_a8(Xq, sx).cpu().numpy()
    for r in range(m):
        ref = a8.gemv_a8(q.codes, g, q.scales, q.zeros, X[r])
        if not np.any(ref):
            assert not np.any(Y[r].astype(np.float32)), r
            continue
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, r


CB_FORMATS = [(3, 32), (3, 64), (3, 128), (4, 32), (4, 64), (4, 128)]
CB_SHAPES = [(3, 384), (37, 4096), (19, 8192), (70, 11008), (260, 1024), (4096, 4096)]


@pytest.mark.parametrize("fmt", CB_FORMATS, ids=lambda f: f"cb{f[0]}g{f[1]}")
@pytest.mark.parametrize("shape", CB_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_codebook_gemv_a8_matches_oracle(gpu, fmt, shape):
    """Per-group codebooks with 8-bit activations (QuantX's non-uniform groups in its W3A8
    configurations): y = s_x * sum C[q] xq against the oracle; repeatable bit for bit, and a
    zero vector gives zeros."""
    qx = gpu
    bits, g = fmt
    n, k = shape
    print(f"codebook a8 gemv {fmt} {shape}", flush=True)
    q = (random_quant(n, k, bits, g, 1, seed=n + k + g) if n * k > 4 * 10**6
         else realistic_quant(n, k, bits, g, 1, seed=n + k + g))
    x = activations(k, seed=k + bits)
    pw = qx.PackedWeight.from_quant(q, device="cuda")
    y = pw.gemv_a8(to_dev(x)).cpu().numpy()
    ref = a8.gemv_a8_codebook(q.codes, g, q.codebook, x)
    assert oracle.normwise_rel_err(y, ref) <= TOL
    assert np.array_equal(y.view(np.uint16), pw.gemv_a8(to_dev(x)).cpu().numpy().view(np.uint16))
    assert not np.any(pw.gemv_a8(to_dev(np.zeros(k, np.float16))).cpu().numpy())


@pytest.mark.parametrize("fmt", [(3, 1, 128), (3, 1, 32), (4, 1, 64), (4, 2, 64)],
                         ids=lambda f: f"b{f[0]}k{f[1]}g{f[2]}")
@pytest.mark.parametrize("shape", [(1, 130, 4096), (3, 300, 1152), (16, 257, 11008), (70, 1000, 2048),
                                   (256, 4096, 1024)], ids=lambda s: f"m{s[0]}_{s[1]}x{s[2]}")
def test_table_gemm_a8_matches_oracle(gpu, fmt, shape):
    """qx_gemm_a8 on codebook and Q4X weights: the int8 codes of qx_quantize_a8 times the table
    entries on the fp16 matrix cores (Q4X: each group's sum scaled by its s in fp32), scaled
    per row, against the per-row oracle of the same quantization."""
    import torch
    qx = gpu
    bits, kind, g = fmt
    m, n, k = shape
    print(f"table a8 gemm {fmt} {shape}", flush=True)
    if kind == qx.QX_Q4X:
        from qx_inputs import q4x as qq
        q = qq.quantize_q4x(qi.weights("t4", 0.0141421, n + k, 0, n, k))
    else:
        q = realistic_quant(n, k, bits, g, kind, seed=n + k + m)
    X = activations(k, seed=k + m, m=m)
    pw = qx.PackedWeight.from_quant(q, device="cuda")
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = pw.gemm_a8(Xq, sx).cpu().numpy()
    for r in range(m):
        if kind == qx.QX_Q4X:
            ref = a8.gemv_a8_q4x(q.codes, q.scales, q.selectors, q.codebook, X[r])
        else:
            ref = a8.gemv_a8_codebook(q.codes, g, q.codebook, X[r])
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, r
    Y2 = pw.gemm_a8(Xq, sx).cpu().numpy()
    assert np.array_equal(Y.view(np.uint16), Y2.view(np.uint16))
    if m > 1:  # a row is the same product whatever else is in the batch
        y0 = pw.gemm_a8(Xq[:1].contiguous(), sx[:1].contiguous()).cpu().numpy()
        assert oracle.normwise_rel_err(y0[0], Y[0].astype(np.float64)) <= TOL


@pytest.mark.parametrize("n,k", [(130, 4096), (300, 11008), (64, 1152)], ids=lambda v: str(v))
def test_q4x_gemm_a8_is_the_gemv_a8_product(gpu, n, k):
    """Q4X with 8-bit activations: qx_gemm_a8 multiplies the exact s * CB[t][q] like
    qx_gemv_a8 (each group's sum of table entries times xq scaled by s in fp32), not W'
    rounded to binary16. A one-hot row (x = a e_j, so xq = 127 e_j) gives one exact product
    per output, which both calls scale in the same order: the same bits, for every group
    and selector the probed columns touch; other rows stay within the bound of the oracle."""
    import torch
    from qx_inputs import q4x as qq
    qx = gpu
    rng = np.random.default_rng(n + k)
    G = k // 64
    s16 = np.float16(rng.uniform(0.3, 1.7, (n, G)) * rng.choice([-1.0, 1.0], (n, G))).view(np.uint16)
    cb = np.sort(rng.standard_normal((4, 16)), axis=1).astype(np.float16).view(np.uint16)
    q = qi.QuantWeight(n, k, 4, 64, qq.Q4X, rng.integers(0, 16, (n, k), dtype=np.uint8), scales=s16,
                       codebook=cb, selectors=rng.integers(0, 4, (n, G), dtype=np.uint8))
    pw = qx.PackedWeight.from_quant(q, device="cuda")
    cols = rng.choice(k, 6, replace=False)
    for j in cols:
        x = np.zeros(k, np.float16)
        x[j] = np.float16(rng.uniform(0.5, 3.0))
        Xq, sx = qx.quantize_a8(to_dev(x[None, :]))
        a = pw.gemm_a8(Xq, sx).cpu().numpy()[0]
        b = pw.gemv_a8(to_dev(x)).cpu().numpy()
        assert np.array_equal(a.view(np.uint16), b.view(np.uint16)), j
    X = activations(k, seed=n, m=5)
    Xq, sx = qx.quantize_a8(to_dev(X))
    Y = pw.gemm_a8(Xq, sx).cpu().numpy()
    for r in range(5):
        ref = a8.gemv_a8_q4x(q.codes, q.scales, q.selectors, q.codebook, X[r])
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, r
        y = pw.gemv_a8(to_dev(X[r])).cpu().numpy()
        assert oracle.normwise_rel_err(Y[r], y.astype(np.float64)) <= TOL, r
