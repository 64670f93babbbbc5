"""Pins of the shared input generator and quantizers (CPU only).

The quantizers produce the codes and fp16 tables that both the oracle and the
HIP path consume, so they are pinned against definitions rather than against
either side: a library Philox, numpy's binary16 rounding, the closed-form
uniform error bound, and brute-force nearest-entry search.
"""
import numpy as np
import pytest

import qx_inputs as qi
from qx_inputs import configs
import oracle


# ------------------------------------------------------------------ generator
@pytest.mark.parametrize("ctr,key", [([0, 0, 0, 0], [0, 0]), ([5, 0, 0, 0], [7, 9]),
                                     ([2**64 - 2, 3, 4, 5], [2**63, 12345])])
def test_philox_matches_numpy_bitgenerator(ctr, key):
    # numpy's Philox advances its counter before producing a block
    bg = np.random.Philox(counter=np.array(ctr, np.uint64), key=np.array(key, np.uint64))
    ref = bg.random_raw(4)
    nxt = list(ctr)
    nxt[0] = (nxt[0] + 1) % 2**64
    assert np.array_equal(qi.philox4x64(nxt, key), ref)


def test_double_to_half_rne_matches_numpy():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(200_000) * 10.0 ** rng.uniform(-9, 5, 200_000),
        np.arange(-70000, 70000, 0.25),
    ])
    # exact ties between neighbouring binary16 values, and the overflow threshold
    h = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    mids = (h[:-1] + h[1:]) / 2
    x = np.concatenate([x, mids, -mids, [65504.0, 65519.99, 65520.0, 1e6, 0.0, -0.0]])
    got = qi.double_to_half_bits(x, 0)
    want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want)


def test_double_to_half_round_up_is_smallest_half_not_below():
    rng = np.random.default_rng(1)
    x = np.abs(rng.standard_normal(100_000)) * 10.0 ** rng.uniform(-9, 4, 100_000)
    up = qi.double_to_half_bits(x, 1).view(np.float16)
    assert np.all(up.astype(np.float64) >= x)
    below = np.nextafter(up, np.float16(0))
    assert np.all(below.astype(np.float64) < x)
    exact = np.float16([0.5, 1.0, 2.0 ** -24, 3.0]).astype(np.float64)
    assert np.array_equal(qi.double_to_half_bits(exact, 1).view(np.float16).astype(np.float64), exact)


def test_rows_regenerate_independently():
    spec, _ = configs.c3()
    full = qi.weights(spec.dist, spec.p, spec.seed, spec.stream, 64, spec.k)
    part = qi.weights(spec.dist, spec.p, spec.seed, spec.stream, 64, spec.k, row0=17, rows=5)
    assert np.array_equal(full[17:22], part)


def test_distribution_moments():
    n = 2_000_000
    z = qi.fill("normal", 1.0, 11, 0, 0, n)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    lap = qi.fill("laplace", 0.008, 11, 1, 0, n)
    assert abs(np.abs(lap).mean() - 0.008) < 1e-4          # E|X| = b
    t = qi.fill("t4", 0.02, 11, 2, 0, n)
    from scipy import stats
    med = stats.t.ppf(0.75, 4) / np.sqrt(2)  # median |t4|, scaled to unit std
    assert abs(np.median(np.abs(t)) / 0.02 - med) < 0.005
    assert np.mean(np.abs(t) > 5 * 0.02) > 10 * np.mean(np.abs(z) > 5)  # heavy tails


def test_outlier_channels():
    spec, x = configs.c2()
    ch = qi.outlier_channels(1, 2, 4096)
    assert len(ch) == 41 and len(set(ch.tolist())) == 41
    base = qi.activations(1, 1, 4096)
    ratio = x[ch].astype(np.float64) / base[ch].astype(np.float64)
    assert np.allclose(ratio, 20, rtol=2e-3)
    others = np.setdiff1d(np.arange(4096), ch)
    assert np.array_equal(x[others], base[others])


# ------------------------------------------------------------------ uniform
def _adversarial_groups(g):
    rng = np.random.default_rng(5)
    rows = [np.zeros(g), np.full(g, 0.37), np.full(g, -0.2), np.abs(rng.standard_normal(g)),
            -np.abs(rng.standard_normal(g)), rng.standard_normal(g) * 1e-6,
            np.r_[rng.standard_normal(g - 1) * 0.01, 5.0], rng.standard_t(4, g) * 0.02,
            np.linspace(-1, 1, g), rng.standard_normal(g) * 1e3]
    return np.array(rows, dtype=np.float32)


@pytest.mark.parametrize("bits,g", [(3, 64), (3, 128), (4, 128), (4, 64), (3, 32)])
def test_uniform_roundtrip_bound(bits, g):
    """|w - s16 (q - z)| <= s16 / 2 per element, and W' adds at most half a binary16 ulp."""
    w = np.concatenate([_adversarial_groups(g).reshape(-1, g),
                        qi.weights("t4", 0.02, 1, 0, 64, 4 * g).reshape(-1, g)]).reshape(-1, g)
    q = qi.quantize_uniform(w, bits, g)
    s = q.scales.view(np.float16).astype(np.float64)[:, 0]
    z = q.zeros.view(np.float16).astype(np.float64)[:, 0]
    assert np.all(z == np.round(z)) and np.all((z >= 0) & (z <= 2**bits - 1))
    assert q.codes.max() < 2**bits
    lev = s[:, None] * (q.codes.astype(np.float64) - z[:, None])
    err = np.abs(w.astype(np.float64) - lev)
    assert np.all(err <= s[:, None] / 2 * (1 + 1e-12))
    # the step is the smallest binary16 not below (max(w,0) - min(w,0)) / (2^b - 1)
    lo = np.minimum(w.min(1), 0).astype(np.float64)
    hi = np.maximum(w.max(1), 0).astype(np.float64)
    raw = (hi - lo) / (2**bits - 1)
    nz = hi > lo
    assert np.all(s[nz] >= raw[nz])
    prev = np.nextafter(s[nz].astype(np.float16), np.float16(0)).astype(np.float64)
    assert np.all(prev < raw[nz])
    assert np.all(s[~nz] == 1.0) and np.all(q.codes[~nz] == 0)
    w16 = oracle.dequant(q.codes, g, 0, q.scales, q.zeros)
    ulp = np.abs(np.spacing(w16.astype(np.float16))).astype(np.float64)
    assert np.all(np.abs(w.astype(np.float64) - w16.astype(np.float64)) <= s[:, None] / 2 * (1 + 1e-12) + ulp / 2)


def test_uniform_codes_are_nearest_level_brute_force():
    g, bits = 16, 3
    w = qi.weights("normal", 0.5, 9, 0, 40, g)
    q = qi.quantize_uniform(w, bits, g)
    s = q.scales.view(np.float16).astype(np.float64)[:, 0]
    z = q.zeros.view(np.float16).astype(np.float64)[:, 0]
    for r in range(w.shape[0]):
        levels = s[r] * (np.arange(2**bits) - z[r])
        d = np.abs(w[r].astype(np.float64)[:, None] - levels[None, :])
        best = d.min(1)
        picked = d[np.arange(g), q.codes[r]]
        assert np.all(picked == best)


# ------------------------------------------------------------------ codebook
@pytest.mark.parametrize("bits,g,dist,p", [(3, 128, "laplace", 0.008), (3, 64, "t4", 0.02),
                                           (4, 128, "laplace", 0.008), (3, 32, "normal", 1.0)])
def test_codebook_codes_are_nearest_entry_brute_force(bits, g, dist, p):
    w = np.concatenate([qi.weights(dist, p, 21, 0, 6, 2 * g), _adversarial_groups(2 * g)[:, :2 * g]])
    w = np.ascontiguousarray(w, dtype=np.float32)
    q = qi.quantize_codebook(w, bits, g)
    n, k = w.shape
    cb = q.codebook.view(np.float16).astype(np.float64)
    assert np.all(np.diff(cb, axis=-1) >= 0), "codebook entries ascending"
    for r in range(n):
        for j in range(k // g):
            vals = w[r, j * g:(j + 1) * g].astype(np.float64)
            d = np.abs(vals[:, None] - cb[r, j][None, :])
            assert np.array_equal(q.codes[r, j * g:(j + 1) * g], np.argmin(d, axis=1))


def test_codebook_lloyd_fixed_point_and_mse():
    g, bits = 128, 3
    w = qi.weights("laplace", 0.008, 22, 0, 32, 4 * g)
    q = qi.quantize_codebook(w, bits, g, keep_raw=True)
    raw, iters = q.meta["raw_centroids"], q.meta["iters"]
    qu = qi.quantize_uniform(w, bits, g)
    wu = oracle.dequant(qu.codes, g, 0, qu.scales, qu.zeros).astype(np.float64)
    for r in range(w.shape[0]):
        for j in range(w.shape[1] // g):
            vals = w[r, j * g:(j + 1) * g].astype(np.float64)
            c = raw[r, j]
            assert np.all(np.diff(c) > 0)
            lab = np.argmin(np.abs(vals[:, None] - c[None, :]), axis=1)
            if iters[r, j] < 100:
                for e in range(2**bits):
                    if np.any(lab == e):
                        assert abs(vals[lab == e].mean() - c[e]) <= 1e-12 * max(1e-3, abs(c[e]))
            mse_cb = np.mean((vals - c[lab]) ** 2)
            mse_u = np.mean((vals - wu[r, j * g:(j + 1) * g]) ** 2)
            assert mse_cb <= mse_u * (1 + 1e-9) + 1e-18
    assert np.mean(iters < 100) > 0.95


def test_codebook_equal_to_uniform_grid_matches_uniform_dequant():
    """A codebook holding the uniform levels s(e - z) dequantizes bit-identically."""
    g, bits = 64, 3
    w = qi.weights("t4", 0.02, 23, 0, 16, 256)
    qu = qi.quantize_uniform(w, bits, g)
    s = qu.scales.view(np.float16).astype(np.float64)
    z = qu.zeros.view(np.float16).astype(np.float64)
    levels = (s[..., None] * (np.arange(2**bits) - z[..., None])).astype(np.float16)
    wu = oracle.dequant(qu.codes, g, 0, qu.scales, qu.zeros)
    wc = oracle.dequant(qu.codes, g, 1, codebook=levels.view(np.uint16))
    assert np.array_equal(wu.view(np.uint16), wc.view(np.uint16))


def test_config_shapes_and_bytes():
    assert configs.c1()[0].packed_bytes == 8_912_896
    assert configs.c2()[0].packed_bytes == 19_726_336
    assert configs.c3()[0].packed_bytes == 8_388_608
    plan = configs.c4_plan()
    assert len(plan) == 224
    assert sum(s.packed_bytes for s, _ in plan) == 3_373_268_992
    assert sum(configs.c5_matrix(m).packed_bytes for m in ("gate", "up", "down")) == 59_179_008
