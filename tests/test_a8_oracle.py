"""Pins of the 8-bit-activation oracle (CPU only): per-token symmetric RTN
(Section 2.4; Table 1's W3A8 configurations) and the integer-domain product of
uniform codes with int8 activations."""
import numpy as np
import pytest

import oracle
from oracle import a8
import qx_inputs as qi


def test_activation_by_hand():
    x = np.float16([0.5, -1.0, 0.25, 2.0, -2.0, 0.0, 1.0 / 3])
    xq, s = a8.quantize_activation(x)
    assert s == np.float32(2.0) / np.float32(127.0)
    # 0.5 * 63.5 = 31.75 -> 32; -1 -> -63.5 -> -64 (ties to even); 0.25 -> 15.875 -> 16
    assert xq.tolist() == [32, -64, 16, 127, -127, 0, 21]


def test_activation_extremes_and_bound():
    x = qi.activations(3, 1, 4096, outliers=np.arange(0, 4096, 97))
    xq, s = a8.quantize_activation(x)
    xf = x.astype(np.float64)
    assert np.abs(xq).max() == 127 and xq[np.argmax(np.abs(xf))] in (127, -127)
    # each code is the nearest integer to x * inv (exact product), so within 1/2 of x / s_x
    # up to the relative rounding of inv and s_x
    _, inv = 0, np.float32(127.0) / np.float32(np.abs(xf).max())
    assert np.all(np.abs(xf * np.float64(inv) - xq) <= 0.5)
    err = np.abs(xf / float(s) - xq.astype(np.float64))
    assert err.max() <= 0.5 + 1e-5
    assert np.all(np.abs(xf - float(s) * xq) <= float(s) * (0.5 + 1e-5))


def test_zero_activation():
    xq, s = a8.quantize_activation(np.zeros(256, np.float16))
    assert s == 0 and not xq.any()
    q = qi.quantize_uniform(qi.weights("t4", 0.02, 1, 2, 4, 256), 4, 64)
    assert not a8.gemv_a8(q.codes, 64, q.scales, q.zeros, np.zeros(256, np.float16)).any()


@pytest.mark.parametrize("bits,group", [(3, 64), (4, 128), (3, 32)])
def test_gemv_a8_brute_force(bits, group):
    rng = np.random.default_rng(bits * group)
    n, k = 5, 256
    q = qi.quantize_uniform(qi.weights("t4", 0.02, 2, bits, n, k), bits, group)
    x = np.float16(rng.standard_normal(k))
    y = a8.gemv_a8(q.codes, group, q.scales, q.zeros, x)
    xq, s_x = a8.quantize_activation(x)
    s = q.scales.view(np.float16).astype(np.float64)
    z = q.zeros.view(np.float16).astype(np.float64)
    for r in range(n):
        tot = 0.0
        for g in range(k // group):
            acc = 0
            for i in range(g * group, (g + 1) * group):
                acc += (int(q.codes[r, i]) - int(z[r, g])) * int(xq[i])
            tot += s[r, g] * acc
        assert y[r] == pytest.approx(float(s_x) * tot, rel=1e-12, abs=1e-12)


def test_gemv_a8_close_to_a16():
    """Quantizing x to 8 bits moves y by at most s_x/2 * sum_k |W'| per row (plus the
    binary16 rounding of W' that the A16 path applies)."""
    n, k = 64, 4096
    q = qi.quantize_uniform(qi.weights("t4", 0.02, 4, 5, n, k), 4, 128)
    x = qi.activations(4, 6, k)
    y8 = a8.gemv_a8(q.codes, 128, q.scales, q.zeros, x)
    w16 = oracle.dequant(q.codes, 128, 0, q.scales, q.zeros).astype(np.float64)
    y16 = w16 @ x.astype(np.float64)
    _, s_x = a8.quantize_activation(x)
    bound = float(s_x) / 2 * np.abs(w16).sum(axis=1) + 2.0**-11 * (np.abs(w16) @ np.abs(x.astype(np.float64)))
    assert np.all(np.abs(y8 - y16) <= bound * (1 + 1e-9))


def test_gemv_a8_q4x_brute_force():
    """Q4X with 8-bit activations: the loops of the definition, entry by entry."""
    rng = np.random.default_rng(5)
    n, k = 4, 192
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    sel = rng.integers(0, 4, (n, G), dtype=np.uint8)
    s = np.float16(rng.uniform(0.5, 2.0, (n, G))).view(np.uint16)
    cb = np.float16(rng.standard_normal((4, 16))).view(np.uint16)
    x = np.float16(rng.standard_normal(k))
    y = a8.gemv_a8_q4x(codes, s, sel, cb, x)
    xq, s_x = a8.quantize_activation(x)
    cbf = cb.view(np.float16).astype(float)
    sf = s.view(np.float16).astype(float)
    for r in range(n):
        tot = 0.0
        for g in range(G):
            acc = 0.0
            for i in range(64 * g, 64 * g + 64):
                acc += cbf[sel[r, g], codes[r, i]] * int(xq[i])
            tot += sf[r, g] * acc
        assert y[r] == pytest.approx(float(s_x) * tot, rel=1e-12, abs=1e-12)


def test_gemv_a8_q4x_reduces_to_uniform_levels():
    """A Q4X matrix whose sub-codebooks hold the integer levels q - z (z per selector) and
    whose scales are the uniform scales gives the uniform A8 result."""
    rng = np.random.default_rng(8)
    n, k = 6, 256
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    zsel = rng.integers(0, 4, (n, G), dtype=np.uint8)     # zero point 4 * selector
    cb = np.stack([np.arange(16) - 4 * t for t in range(4)]).astype(np.float16).view(np.uint16)
    s = np.float16(rng.uniform(0.01, 0.1, (n, G)))
    x = np.float16(rng.standard_normal(k))
    y = a8.gemv_a8_q4x(codes, s.view(np.uint16), zsel, cb, x)
    z = (4 * zsel).astype(np.float16)
    yu = a8.gemv_a8(codes, 64, s.view(np.uint16), z.view(np.uint16), x)
    assert np.allclose(y, yu, rtol=1e-12, atol=1e-12)


# ---- per-group codebooks with 8-bit activations

@pytest.mark.parametrize("bits,group", [(3, 128), (3, 32), (4, 64)])
def test_gemv_a8_codebook_brute_force(bits, group):
    rng = np.random.default_rng(bits + group)
    n, k = 4, 256
    q = qi.quantize_codebook(qi.weights("laplace", 0.008, 5, bits, n, k), bits, group)
    x = np.float16(rng.standard_normal(k))
    y = a8.gemv_a8_codebook(q.codes, group, q.codebook, x)
    xq, s_x = a8.quantize_activation(x)
    cb = q.codebook.reshape(n, k // group, 1 << bits).view(np.float16)
    for r in range(n):
        tot = 0.0
        for i in range(k):
            tot += float(cb[r, i // group, q.codes[r, i]]) * int(xq[i])
        assert y[r] == pytest.approx(float(s_x) * tot, rel=1e-12, abs=1e-15)


def test_gemv_a8_codebook_reduces_to_uniform():
    """Tables holding the uniform levels s (q - z) (exact in binary16 for a power-of-two s)
    give the integer-domain uniform result exactly."""
    rng = np.random.default_rng(3)
    n, k, bits, group = 6, 512, 3, 64
    G = k // group
    codes = rng.integers(0, 8, (n, k)).astype(np.uint8)
    z = rng.integers(0, 8, (n, G))
    s = 2.0 ** rng.integers(-12, -4, (n, G))
    levels = s[:, :, None] * (np.arange(8)[None, None, :] - z[:, :, None])
    cb = levels.astype(np.float16).view(np.uint16)
    assert np.array_equal(cb.view(np.float16).astype(np.float64), levels)  # the levels are exact
    x = np.float16(rng.standard_normal(k))
    y_cb = a8.gemv_a8_codebook(codes, group, cb, x)
    y_u = a8.gemv_a8(codes, group, s.astype(np.float16).view(np.uint16), z.astype(np.float16).view(np.uint16), x)
    assert np.allclose(y_cb, y_u, rtol=1e-14, atol=0)


def test_gemv_a8_codebook_error_bound():
    """Against the fp16-activation product of the same W': |y_a8 - W' x| <= sum |W'| s_x / 2 per
    row (each xq is within half a step of x / s_x), up to the rounding of s_x."""
    n, k, bits, group = 20, 1024, 3, 128
    q = qi.quantize_codebook(qi.weights("laplace", 0.008, 6, 1, n, k), bits, group)
    x = qi.activations(6, 2, k, outliers=np.arange(0, k, 101))
    w = oracle.dequant(q.codes, group, 1, codebook=q.codebook).astype(np.float64)
    y = a8.gemv_a8_codebook(q.codes, group, q.codebook, x)
    _, s_x = a8.quantize_activation(x)
    bound = np.abs(w).sum(axis=1) * float(s_x) * (0.5 + 1e-5)
    assert np.all(np.abs(y - w @ x.astype(np.float64)) <= bound)


def test_a8_reading_against_plain_rtn_on_the_workloads():
    """The 8-bit activation codes are rint(x * fp32(127/amax)) with the product exact (the
    kernels' arithmetic); plain round-to-nearest of x / (amax/127) in fp64 can differ only
    where x*127/amax lies within an fp32 rounding of a half-integer. On c2 (outlier channels)
    and the first 8 layers' decode-step activations the two readings differ in at most 1 in
    1000 codes of a vector, each by 1 (none on c2)."""
    from qx_inputs import configs
    vectors = [configs.c2()[1]] + [configs.c4_activation(l, t) for l in range(8) for t in range(4)]
    total = 0
    for x in vectors:
        xq, _ = a8.quantize_activation(x)
        amax = np.max(np.abs(x.astype(np.float64)))
        rtn = np.clip(np.rint(x.astype(np.float64) / (amax / 127.0)), -127, 127).astype(np.int64)
        d = np.abs(xq.astype(np.int64) - rtn)
        assert d.max() <= 1 and int(np.sum(d)) <= x.size // 1000
        if x is vectors[0]:
            assert not d.any()  # c2
        total += int(np.sum(d))
    print(f"codes differing from plain RTN: {total} of {sum(v.size for v in vectors)}")
