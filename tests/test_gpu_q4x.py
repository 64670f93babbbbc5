"""Parity of the Q4X path (through the C ABI) with the fp64 oracle.

Q4X (Section 3.2, Q4X item): per-matrix 4 x 16 binary16 codebook; per group of
64 a binary16 scale and a 2-bit sub-codebook selector; W' = fp16_RNE(s *
CB[sel][q]). Dequantized codes and fp16 weights must be bit-exact (including
subnormal and overflowing products); GEMV outputs must satisfy the normwise
bound of the other formats; a one-hot activation must give a column of W' bit
for bit; repeated runs are bitwise identical.
"""
import numpy as np
import pytest

import oracle
from oracle import q4x
import qx_inputs as qi
from qx_inputs import q4x as qq
from helpers import TOL, activations, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(1, 128), (3, 384), (37, 256), (9, 1152), (5, 11008), (130, 4096)]
GEMV_SHAPES = SHAPES + [(33, 12288), (9, 16384), (260, 1024), (19, 8192), (1001, 11008), (4096, 4096)]


def random_q4x(n, k, seed, scale_bits=None):
    """Uniformly random codes, selectors and tables (every code, selector and entry used)."""
    rng = np.random.default_rng(seed)
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    sel = rng.integers(0, 4, (n, G), dtype=np.uint8)
    if scale_bits is None:
        s = np.float16(rng.uniform(0.25, 2.0, (n, G)) * rng.choice([-1.0, 1.0], (n, G), p=[0.1, 0.9]))
        scale_bits = s.view(np.uint16)
    cb = np.sort(rng.standard_normal((4, 16)) * 0.5, axis=1).astype(np.float16).view(np.uint16)
    return qi.QuantWeight(n, k, 4, 64, qq.Q4X, codes, scales=scale_bits, codebook=cb, selectors=sel)


def realistic_q4x(n, k, seed):
    return qq.quantize_q4x(qi.weights("t4", 0.0141421, seed, 0, n, k))


def _ref(q):
    return q4x.dequant(q.codes, q.scales, q.selectors, q.codebook)


def _pack(qx, q):
    return qx.PackedWeight.from_quant(q)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_q4x_dequant_bit_exact(gpu, shape):
    qx = gpu
    n, k = shape
    print(f"q4x dequant {shape}", flush=True)
    q = random_q4x(n, k, seed=n * 13 + k)
    pw = _pack(qx, q)
    assert np.array_equal(pw.dequant(qx.QX_OUT_CODES).cpu().numpy(), q.codes)
    w = pw.dequant(qx.QX_OUT_F16).cpu().numpy()
    assert np.array_equal(w.view(np.uint16), _ref(q).view(np.uint16))


def test_q4x_dequant_full_range_products(gpu):
    """Scales and centroids over the whole finite binary16 range: subnormal results, exact
    zeros of both signs and products that overflow to infinity must all match."""
    qx = gpu
    n, k = 16, 2048
    rng = np.random.default_rng(17)
    G = k // 64
    q = random_q4x(n, k, seed=17)
    q.scales = (rng.integers(0, 0x7C00, (n, G), dtype=np.uint16) |
                (rng.integers(0, 2, (n, G), dtype=np.uint16) << 15))
    q.codebook = (rng.integers(0, 0x7C00, (4, 16), dtype=np.uint16) |
                  (rng.integers(0, 2, (4, 16), dtype=np.uint16) << 15))
    q.codebook[0, :4] = [0x0000, 0x8000, 0x0001, 0x8001]  # zeros and the smallest subnormals
    w = _pack(qx, q).dequant(qx.QX_OUT_F16).cpu().numpy()
    ref = _ref(q)
    assert np.array_equal(w.view(np.uint16), ref.view(np.uint16))
    assert np.isinf(ref.astype(np.float32)).any() and (np.abs(ref.astype(np.float32)) < 2.0**-14).any()


@pytest.mark.parametrize("shape", GEMV_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_q4x_gemv_matches_oracle(gpu, shape):
    qx = gpu
    n, k = shape
    print(f"q4x gemv {shape}", flush=True)
    q = realistic_q4x(n, k, seed=n + k)
    x = activations(k, seed=k + 4)
    y = _pack(qx, q).gemv(to_dev(x)).cpu().numpy()
    err = oracle.normwise_rel_err(y, oracle.gemv(_ref(q), x))
    print(f"  normwise rel err {err:.2e}")
    assert err <= TOL, err


@pytest.mark.parametrize("k", [128, 1152, 4096, 11008, 16384])
def test_q4x_gemv_one_hot_zero_and_determinism(gpu, k):
    qx = gpu
    n = 70
    q = random_q4x(n, k, seed=k)
    pw = _pack(qx, q)
    w16 = _ref(q)
    for j in (0, 63, 64, k // 2 + 5, k - 1):
        x = np.zeros(k, np.float16)
        x[j] = 1.0
        y = pw.gemv(to_dev(x)).cpu().numpy()
        assert np.array_equal(y.view(np.uint16), w16[:, j].view(np.uint16)), j
    assert np.all(pw.gemv(to_dev(np.zeros(k, np.float16))).cpu().numpy() == 0)
    xd = to_dev(activations(k, seed=3))
    a = pw.gemv(xd).cpu().numpy()
    b = pw.gemv(xd).cpu().numpy()
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


def test_q4x_max_k(gpu):
    qx = gpu
    k = 1 << 20
    print("q4x k = 2^20", flush=True)
    q = random_q4x(3, k, seed=21)
    pw = _pack(qx, q)
    w16 = _ref(q)
    assert np.array_equal(pw.dequant(qx.QX_OUT_F16).cpu().numpy().view(np.uint16), w16.view(np.uint16))
    x = activations(k, seed=7)
    assert oracle.normwise_rel_err(pw.gemv(to_dev(x)).cpu().numpy(), oracle.gemv(w16, x)) <= TOL


GEMM_CASES = [(1, 40, 1152), (2, 40, 1152), (3, 130, 4096), (4, 4096, 4096), (2, 11008, 4096),
              (4, 300, 11008), (16, 100, 384), (17, 37, 11008), (64, 300, 1024), (65, 64, 4096),
              (512, 260, 2048), (9, 130, 11008)]


@pytest.mark.parametrize("m,n,k", GEMM_CASES, ids=lambda v: str(v))
def test_q4x_gemm_matches_oracle(gpu, m, n, k):
    """qx_gemm on Q4X (m = 1: the GEMV; m = 2-4: the small-batch kernel; else the
    matrix-core GEMM with W' decoded into its operands as fp16(s * CB[t][q])): every
    output row within the parity bound."""
    qx = gpu
    print(f"q4x gemm m={m} {n}x{k}", flush=True)
    q = random_q4x(n, k, seed=m * 7 + n) if m % 2 or n * k > 10**7 else realistic_q4x(n, k, seed=m + n)
    X = activations(k, seed=m + 3, m=m)
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    w = _ref(q)
    for r in range(m):
        assert oracle.normwise_rel_err(Y[r], oracle.gemv(w, X[r])) <= TOL, r


def test_q4x_gemm_one_hot_rows_are_columns_of_w(gpu):
    """Each activation row one-hot at a different position: the product is exact, so row r
    of Y is column j_r of W' bit for bit, zeros up to sign (checks the fragment decode,
    scales and selectors of every group the rows touch)."""
    qx = gpu
    n, k, m = 64, 4096, 64
    q = random_q4x(n, k, seed=11)
    cols = np.random.default_rng(3).choice(k, m, replace=False)
    X = np.zeros((m, k), np.float16)
    X[np.arange(m), cols] = 1.0
    Y = _pack(qx, q).gemm(to_dev(X)).cpu().numpy()
    w = _ref(q)
    ref = w[:, cols].T.copy()
    assert np.array_equal(Y.astype(np.float32), ref.astype(np.float32))  # +0 sums of a -0 weight
    nz = ref.astype(np.float32) != 0
    assert np.array_equal(Y.view(np.uint16)[nz], ref.view(np.uint16)[nz])


@pytest.mark.parametrize("shape", [(40, 1152), (130, 4096), (300, 11008), (4096, 4096), (37, 8192)],
                         ids=lambda s: f"{s[0]}x{s[1]}")
def test_q4x_gemv_a8_matches_oracle(gpu, shape):
    """The paper's Q4X with 8-bit per-token activations (Table 2's configuration)."""
    from oracle import a8
    qx = gpu
    n, k = shape
    q = random_q4x(n, k, seed=n + k) if n * k > 10**7 else realistic_q4x(n, k, seed=n + k)
    x = activations(k, seed=k + 1)
    pw = _pack(qx, q)
    y = pw.gemv_a8(to_dev(x)).cpu().numpy()
    ref = a8.gemv_a8_q4x(q.codes, q.scales, q.selectors, q.codebook, x)
    assert oracle.normwise_rel_err(y, ref) <= TOL
    assert np.array_equal(y.view(np.uint16), pw.gemv_a8(to_dev(x)).cpu().numpy().view(np.uint16))
    assert not np.any(pw.gemv_a8(to_dev(np.zeros(k, np.float16))).cpu().numpy())
