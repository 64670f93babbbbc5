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
from helpers import TOL, activations, realistic_quant, to_dev

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
