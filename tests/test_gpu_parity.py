"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Dequantized codes and fp16 weights must be bit-exact. GEMV/GEMM outputs must
satisfy max|y - y_ref| / max|y_ref| <= 2e-3 per output vector (fp32
accumulation against fp64); one-hot activations must reproduce a column of
W' bit-exactly, and repeated runs must be bitwise identical.
"""
import itertools

import numpy as np
import pytest

import oracle
from qx_inputs import configs
from helpers import TOL, activations, random_quant, realistic_quant, to_dev

pytestmark = pytest.mark.gpu

FORMATS = [(b, kind, g) for b in (3, 4) for kind in (0, 1) for g in (32, 64, 128)]
SHAPES = [(1, 128), (3, 384), (37, 256), (5, 11008), (130, 4096)]


def _fmt_id(f):
    return f"b{f[0]}{'u' if f[1] == 0 else 'c'}g{f[2]}"


def _ref_w16(q):
    return oracle.dequant(q.codes, q.group, q.kind, q.scales, q.zeros, q.codebook)


def _pack(qx, q):
    return qx.PackedWeight.from_quant(q)


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_dequant_bit_exact(gpu, fmt, shape):
    qx = gpu
    bits, kind, g = fmt
    n, k = shape
    print(f"dequant {fmt} {shape}", flush=True)
    q = random_quant(n, k, bits, g, kind, seed=n * 7 + k + bits)
    pw = _pack(qx, q)
    codes = pw.dequant(qx.QX_OUT_CODES).cpu().numpy()
    assert np.array_equal(codes, q.codes)
    w16 = pw.dequant(qx.QX_OUT_F16).cpu().numpy()
    assert np.array_equal(w16.view(np.uint16), _ref_w16(q).view(np.uint16))


def test_dequant_tiny_scales_give_subnormal_halves(gpu):
    qx = gpu
    q = random_quant(4, 256, 3, 64, 0, seed=5, scale_range=(2.0**-24, 2.0**-16))
    w16 = _pack(qx, q).dequant(qx.QX_OUT_F16).cpu().numpy()
    ref = _ref_w16(q)
    assert np.any((ref != 0) & (np.abs(ref.astype(np.float64)) < 2.0**-14))
    assert np.array_equal(w16.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("make", [configs.c1, configs.c2, configs.c3], ids=["c1", "c2", "c3"])
def test_dequant_configs_bit_exact(gpu, make):
    qx = gpu
    spec, _ = make()
    print(f"dequant {spec.name}", flush=True)
    q = spec.quantized()
    pw = _pack(qx, q)
    assert np.array_equal(pw.dequant(qx.QX_OUT_CODES).cpu().numpy(), q.codes)
    w16 = pw.dequant(qx.QX_OUT_F16).cpu().numpy()
    assert np.array_equal(w16.view(np.uint16), _ref_w16(q).view(np.uint16))


# covers every GEMV kernel path: rows of 32 or 64 chunks (in-wave reduction), rows of
# up to 88 chunks (one chunk per lane), longer rows (K tiles), ragged row counts
GEMV_SHAPES = SHAPES + [(33, 12288), (9, 16384), (260, 1024), (19, 8192), (1001, 11008),
                        (300, 512), (70, 1408)]  # 8-way shards of o (k 512) and down (k 11 chunks)


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("shape", GEMV_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_gemv_matches_oracle(gpu, fmt, shape):
    qx = gpu
    bits, kind, g = fmt
    n, k = shape
    print(f"gemv {fmt} {shape}", flush=True)
    q = realistic_quant(n, k, bits, g, kind, seed=n + k)
    x = activations(k, seed=k + bits)
    pw = _pack(qx, q)
    y = pw.gemv(to_dev(x)).cpu().numpy()
    ref = oracle.gemv(_ref_w16(q), x)
    err = oracle.normwise_rel_err(y, ref)
    print(f"gemv {fmt} {shape} normwise rel err {err:.3e}")
    assert err <= TOL, err


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
def test_gemv_one_hot_zero_and_determinism(gpu, fmt):
    qx = gpu
    bits, kind, g = fmt
    n, k = 70, 11008
    q = random_quant(n, k, bits, g, kind, seed=bits * 10 + kind + g)
    pw = _pack(qx, q)
    w16 = _ref_w16(q)
    for j in (0, 1, 47, 48, 95, 96, 127, 5000, k - 1):
        x = np.zeros(k, np.float16)
        x[j] = 1.0
        y = pw.gemv(to_dev(x)).cpu().numpy()
        # exact in value: a sum that starts at +0 cannot return -0, so -0 entries of W'
        # (negative scale, q == z) come back as +0; every nonzero entry must match bit for bit
        assert np.array_equal(y.astype(np.float64), w16[:, j].astype(np.float64)), j
    y0 = pw.gemv(to_dev(np.zeros(k, np.float16))).cpu().numpy()
    assert np.all(y0 == 0)
    x = activations(k, seed=3)
    xd = to_dev(x)
    a = pw.gemv(xd).cpu().numpy()
    b = pw.gemv(xd).cpu().numpy()
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


@pytest.mark.parametrize("make", [configs.c1, configs.c2, configs.c3], ids=["c1", "c2", "c3"])
def test_gemv_configs(gpu, make):
    qx = gpu
    spec, x = make()
    print(f"gemv {spec.name}", flush=True)
    q = spec.quantized()
    pw = _pack(qx, q)
    y = pw.gemv(to_dev(x)).cpu().numpy()
    ref = oracle.gemv(_ref_w16(q), x)
    err = oracle.normwise_rel_err(y, ref)
    print(f"{spec.name} normwise rel err {err:.3e}")
    assert err <= TOL, err


GEMM_M = [1, 2, 3, 4, 5, 16, 17, 33, 64, 65]


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("m", GEMM_M)
def test_gemm_matches_oracle(gpu, fmt, m):
    qx = gpu
    bits, kind, g = fmt
    n, k = 100, 384
    print(f"gemm {fmt} m={m}", flush=True)
    q = realistic_quant(n, k, bits, g, kind, seed=m + bits)
    X = activations(k, seed=m, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    ref = oracle.gemm(X, _ref_w16(q))
    for r in range(m):
        assert oracle.normwise_rel_err(Y[r], ref[r]) <= TOL, r


SMALL_BATCH = [(4096, 4096), (11008, 4096), (4096, 11008), (37, 1152), (9, 128), (130, 8192)]


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
@pytest.mark.parametrize("m", [2, 3, 4])
@pytest.mark.parametrize("shape", SMALL_BATCH, ids=lambda s: f"{s[0]}x{s[1]}")
def test_gemm_small_batch(gpu, fmt, m, shape):
    """2 <= m <= 4: the GEMV-style small-batch kernel (every code decoded once and
    multiplied with each activation row) where the library routes it (m = 2, or k > n),
    else the matrix-core GEMM; rows of the oracle one by one."""
    qx = gpu
    bits, kind, g = fmt
    n, k = shape
    print(f"gemm small batch {fmt} {shape} m={m}", flush=True)
    q = random_quant(n, k, bits, g, kind, seed=n + k + m) if n * k > 10**7 else \
        realistic_quant(n, k, bits, g, kind, seed=n + k + m)
    X = activations(k, seed=m + 5, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    w16 = _ref_w16(q)
    rows = np.arange(n) if n <= 4096 else np.sort(np.random.default_rng(m).choice(n, 2048, replace=False))
    for r in range(m):
        ref = oracle.gemv(w16[rows], X[r])
        assert oracle.normwise_rel_err(Y[r][rows], ref) <= TOL, r


@pytest.mark.parametrize("m", [2, 4])
def test_gemm_small_batch_longest_k(gpu, m):
    """k = 2^20 (8192 chunks, 256 segments of the small-batch kernel), rows of the oracle."""
    qx = gpu
    n, k = 5, 1 << 20
    q = random_quant(n, k, 4, 128, 0, seed=m)
    X = activations(k, seed=m + 11, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    w16 = _ref_w16(q)
    for r in range(m):
        assert oracle.normwise_rel_err(Y[r], oracle.gemv(w16, X[r])) <= TOL, r


@pytest.mark.parametrize("fmt", [(4, 0, 128), (4, 1, 32)], ids=_fmt_id)
def test_gemm_one_row_is_the_gemv(gpu, fmt):
    """m = 1 runs the batch-1 GEMV: the same bits as qx_gemv (the 4-bit codebook of
    32-code groups too, on rows of 32 chunks)."""
    qx = gpu
    bits, kind, g = fmt
    q = realistic_quant(300, 4096, bits, g, kind, seed=4)
    pw = _pack(qx, q)
    x = activations(4096, seed=2)
    a = pw.gemm(to_dev(x[None, :])).cpu().numpy()[0]
    b = pw.gemv(to_dev(x)).cpu().numpy()
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


@pytest.mark.parametrize("m", [16, 32, 64, 128, 256, 512])
@pytest.mark.parametrize("name", ["gate", "down"])
def test_gemm_prefill_shapes(gpu, m, name):
    """c5 matrices; down at m = 32 / 128 / 256 takes the k split over more waves."""
    qx = gpu
    spec = configs.c5_matrix(name)
    print(f"gemm c5 {name} m={m}", flush=True)
    q = spec.quantized()
    xin, xdn = configs.c5_activations(m)
    X = xdn if name == "down" else xin
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    rows = range(m) if m <= 64 else range(0, m, 37)
    w16 = _ref_w16(q)
    for r in rows:
        ref = oracle.gemv(w16, X[r])
        assert oracle.normwise_rel_err(Y[r], ref) <= TOL, r


# activation tiles mapped to XCDs with padding blocks, single-chunk rows, chunk counts
# that leave K-split waves idle in the last round; 128 x 192 blocks (uniform formats at
# m >= 384) with ragged weight and activation rows; 128 x 256 blocks of 8 waves where those
# take fewer rounds (11000 rows at m = 600: last block of 248 rows, last tile of 88; 16400
# rows at m = 384)
GEMM_EDGES = [(40, 1024, 300), (300, 1152, 100), (17, 128, 129), (70, 640, 40), (1, 640, 17),
              (4096, 1152, 128), (2000, 1536, 200), (9601, 1152, 390), (4800, 640, 768),
              (11000, 640, 600), (16400, 384, 384)]


@pytest.mark.parametrize("fmt", [(3, 0, 64), (4, 0, 128), (3, 1, 32), (4, 1, 32)], ids=_fmt_id)
@pytest.mark.parametrize("shape", GEMM_EDGES, ids=lambda s: f"{s[0]}x{s[1]}m{s[2]}")
def test_gemm_tile_edges(gpu, fmt, shape):
    qx = gpu
    bits, kind, g = fmt
    n, k, m = shape
    print(f"gemm {fmt} {shape}", flush=True)
    q = realistic_quant(n, k, bits, g, kind, seed=n + k + m)
    X = activations(k, seed=m + 1, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    ref = oracle.gemm(X, _ref_w16(q))
    for r in range(m):
        assert oracle.normwise_rel_err(Y[r], ref[r]) <= TOL, r


def test_gemm_rows_equal_gemv_within_tolerance(gpu):
    qx = gpu
    q = realistic_quant(257, 1024, 3, 64, 0, seed=11)
    X = activations(1024, seed=12, m=9)
    pw = _pack(qx, q)
    Y = pw.gemm(to_dev(X)).cpu().numpy()
    for r in range(9):
        y = pw.gemv(to_dev(X[r])).cpu().numpy()
        assert oracle.normwise_rel_err(Y[r], y.astype(np.float64)) <= 2 * TOL


@pytest.mark.parametrize("fmt", [(3, 0, 64), (4, 0, 128), (3, 1, 128), (4, 1, 32)], ids=_fmt_id)
@pytest.mark.parametrize("m", [33, 64, 256, 512])
def test_gemm_long_rows_wide_split(gpu, fmt, m):
    """Rows of more than 64 chunks with the k split over 8 waves: at 16 < m <= 64 with enough
    weight rows that uniform 32 x 32 tiles number more than 128, and at m = 256 / 512 with
    129-256 tiles (sampled rows against the oracle)."""
    qx = gpu
    bits, kind, g = fmt
    n, k = (4200 if m <= 64 else 4096), 11008
    print(f"gemm long rows {fmt} m={m}", flush=True)
    q = random_quant(n, k, bits, g, kind, seed=m + g)
    X = activations(k, seed=m + 3, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    rows = sorted(set(range(0, m, 1 if m <= 64 else 29)) | {m - 1})
    ref = oracle.gemm(X[rows], _ref_w16(q))
    for i, r in enumerate(rows):
        assert oracle.normwise_rel_err(Y[r], ref[i]) <= TOL, r


# ---- maximum sizes and degenerate inputs

K_MAX = 1 << 20  # largest k the interface accepts
EDGE_FORMATS = [(3, 0, 64), (4, 0, 128), (3, 1, 128), (4, 1, 32)]


@pytest.mark.parametrize("fmt", EDGE_FORMATS, ids=_fmt_id)
def test_max_k_dequant_and_gemv(gpu, fmt):
    qx = gpu
    bits, kind, g = fmt
    print(f"k = 2^20 {fmt}", flush=True)
    q = random_quant(3, K_MAX, bits, g, kind, seed=bits + g)
    pw = _pack(qx, q)
    w16 = _ref_w16(q)
    assert np.array_equal(pw.dequant(qx.QX_OUT_CODES).cpu().numpy(), q.codes)
    assert np.array_equal(pw.dequant(qx.QX_OUT_F16).cpu().numpy().view(np.uint16), w16.view(np.uint16))
    x = activations(K_MAX, seed=7)
    y = pw.gemv(to_dev(x)).cpu().numpy()
    assert oracle.normwise_rel_err(y, oracle.gemv(w16, x)) <= TOL
    X = activations(K_MAX, seed=8, m=3)
    Y = pw.gemm(to_dev(X)).cpu().numpy()
    ref = oracle.gemm(X, w16)
    for r in range(3):
        assert oracle.normwise_rel_err(Y[r], ref[r]) <= TOL, r


def test_max_m_gemm(gpu):
    qx = gpu
    m, n, k = 65536, 20, 256  # the largest m the interface accepts
    print("gemm m = 65536", flush=True)
    q = realistic_quant(n, k, 3, 64, 0, seed=3)
    X = activations(k, seed=9, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    ref = oracle.gemm(X, _ref_w16(q))
    err = max(oracle.normwise_rel_err(Y[r], ref[r]) for r in range(0, m, 97))
    assert err <= TOL, err
    assert oracle.normwise_rel_err(Y[m - 1], ref[m - 1]) <= TOL


@pytest.mark.parametrize("fmt", FORMATS, ids=_fmt_id)
def test_zero_weights_give_zero(gpu, fmt):
    """Every code at the zero point (uniform) or every table entry +0 (codebook): W' = 0
    exactly. Dequant and GEMM (which multiply W') give exact zeros. The uniform GEMV folds
    the zero point out per group, s * (sum (M+q) x - sum M x - z sum x), so its zero comes
    out of fp32 rounding of those sums: bounded here by 2e-3 of what one code step per
    weight gives, sum_k |s| |x_k|, per row (the normwise scale of the parity bound)."""
    qx = gpu
    bits, kind, g = fmt
    n, k = 70, 11008
    q = random_quant(n, k, bits, g, kind, seed=17)
    if kind == 0:
        zi = np.random.default_rng(1).integers(0, 2**bits, (n, k // g))
        q.zeros = zi.astype(np.float16).view(np.uint16)
        q.codes = np.repeat(zi, g, axis=1).astype(np.uint8)
    else:
        q.codebook = np.zeros_like(q.codebook)
    pw = _pack(qx, q)
    assert not np.any(pw.dequant(qx.QX_OUT_F16).cpu().numpy().astype(np.float64))
    x = activations(k, seed=2)
    y = pw.gemv(to_dev(x)).cpu().numpy().astype(np.float64)
    if kind == 0:
        s = np.abs(q.scales.view(np.float16).astype(np.float64))
        scale = (s * np.abs(x.astype(np.float64)).reshape(k // g, g).sum(axis=1)).sum(axis=1)
        assert np.all(np.abs(y) <= TOL * scale), np.max(np.abs(y) / scale)
    else:
        assert not np.any(y)
    X = activations(k, seed=3, m=5)
    assert not np.any(pw.gemm(to_dev(X)).cpu().numpy().astype(np.float64))
