"""Pins of the Q4X oracle and quantizer (CPU only).

Q4X (Section 3.2, Q4X item; Figure 3 captions): a per-matrix codebook of 64
binary16 centroids in 4 sub-codebooks of 16; per group of 64 weights a binary16
scale, a 2-bit selector and 64 4-bit indices; W' = fp16_RNE(s * CB[sel][q]).
The pins: the paper's printed bits per weight, hand-derived layout bytes,
pack/unpack identity, a reduction to the per-group codebook oracle, numpy's
binary16 product, and brute force over every level and sub-codebook for the
quantizer's choices.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import q4x
import qx_inputs as qi
from qx_inputs import q4x as qq

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_bits_per_weight_matches_the_paper():
    """Rows with a multiple of 16 groups carry exactly 4 + 18/64 bits per weight; the paper
    prints 4.28 for Q4X (Section 3.2 and Table 2)."""
    printed = [f for f in _load("paper_bpw.json")["formats"] if f["name"] == "Q4X"][0]["printed_bpw"]
    n, k = 4096, 4096
    per_rows = q4x.packed_size(n, k) - 128  # the per-matrix codebook is not per weight
    bpw = per_rows * 8 / (n * k)
    assert bpw == 4 + 18 / 64
    assert round(bpw, 2) == printed


@pytest.mark.parametrize("ex", _load("q4x_layout_examples.json")["examples"], ids=lambda e: e["name"])
def test_layout_worked_examples(ex):
    n, k = ex["n"], ex["k"]
    G = k // 64
    codes = np.zeros((n, k), np.uint8)
    scales = np.zeros((n, G), np.uint16)
    sel = np.zeros((n, G), np.uint8)
    cb = np.zeros((4, 16), np.uint16)
    for r, c, v in ex["codes"]:
        codes[r, c] = v
    for r, j, v in ex["scales"]:
        scales[r, j] = v
    for r, j, v in ex["selectors"]:
        sel[r, j] = v
    for t, e, v in ex["codebook"]:
        cb[t, e] = v
    blob = q4x.pack(codes, scales, sel, cb)
    assert blob.size == ex["size"] == q4x.packed_size(n, k)
    want = np.zeros(ex["size"], np.uint8)
    for off, val in ex["nonzero"].items():
        want[int(off)] = val
    assert np.array_equal(blob, want)
    back = q4x.unpack(blob, n, k)
    for a, b in zip(back, (codes, scales, sel, cb)):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("n,k", [(1, 128), (3, 256), (5, 1152), (2, 11008), (7, 4096)])
def test_pack_unpack_identity(n, k):
    rng = np.random.default_rng(n * 7919 + k)
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    scales = rng.integers(0, 2**16, (n, G), dtype=np.uint16)
    sel = rng.integers(0, 4, (n, G), dtype=np.uint8)
    cb = rng.integers(0, 2**16, (4, 16), dtype=np.uint16)
    blob = q4x.pack(codes, scales, sel, cb)
    assert blob.size == q4x.packed_size(n, k)
    back = q4x.unpack(blob, n, k)
    for a, b in zip(back, (codes, scales, sel, cb)):
        assert np.array_equal(a, b)
    # the codes region is the general 4-bit layout, byte for byte
    ref = oracle.pack(codes, 4, 128, 0, scales=np.zeros((n, k // 128), np.uint16),
                      zeros=np.zeros((n, k // 128), np.uint16))
    assert np.array_equal(blob[:n * k // 2], ref[:n * k // 2])


def test_unused_selector_bits_are_zero():
    n, k = 3, 1152  # 18 groups: word 1 of each row holds 2 selectors and 28 zero bits
    sel = np.full((n, 18), 3, np.uint8)
    blob = q4x.pack(np.zeros((n, k), np.uint8), np.zeros((n, 18), np.uint16), sel,
                    np.zeros((4, 16), np.uint16))
    l0 = n * k // 2 + n * 18 * 2
    words = blob[l0:l0 + n * 2 * 4].view("<u4").reshape(n, 2)
    assert np.all(words[:, 0] == 0xFFFFFFFF) and np.all(words[:, 1] == 0xF)


def test_dequant_with_unit_scales_is_the_per_group_codebook():
    """s = 1: W' is the selected sub-codebook entry, exactly the per-group codebook path of
    the general oracle with each group's table set to CB[sel]."""
    rng = np.random.default_rng(3)
    n, k = 4, 512
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    sel = rng.integers(0, 4, (n, G), dtype=np.uint8)
    cb = np.float16(rng.standard_normal((4, 16))).view(np.uint16)
    ones = np.full((n, G), 0x3C00, np.uint16)
    w = q4x.dequant(codes, ones, sel, cb)
    per_group = cb[sel]  # [n][G][16]
    ref = oracle.dequant(codes, 64, 1, codebook=per_group)
    assert np.array_equal(w.view(np.uint16), ref.view(np.uint16))


def test_dequant_is_numpys_binary16_product():
    """fp16 x fp16 products are exact in fp32, so numpy's float16 multiply rounds the exact
    product once: it must equal the oracle's fp64 product rounded to binary16, for every
    scale / centroid pair drawn here (normal, subnormal and large values)."""
    rng = np.random.default_rng(5)
    n, k = 8, 1024
    G = k // 64
    codes = rng.integers(0, 16, (n, k), dtype=np.uint8)
    sel = rng.integers(0, 4, (n, G), dtype=np.uint8)
    bits = rng.integers(0, 0x7C00, (n, G), dtype=np.uint16) | (rng.integers(0, 2, (n, G), dtype=np.uint16) << 15)
    cb = (rng.integers(0, 0x7C00, (4, 16), dtype=np.uint16) | (rng.integers(0, 2, (4, 16), dtype=np.uint16) << 15))
    w = q4x.dequant(codes, bits, sel, cb)
    j = np.arange(k) // 64
    s = bits.view(np.float16)[:, j]
    c = cb.view(np.float16)[sel[:, j], codes]
    with np.errstate(over="ignore"):
        ref = (s * c).astype(np.float16)
    assert np.array_equal(w.view(np.uint16), ref.view(np.uint16))


# ------------------------------------------------------------------ quantizer
@pytest.fixture(scope="module")
def small_q4x():
    w = qi.weights("t4", 0.0141421, 4, 9, 6, 512)
    return w, qq.quantize_q4x(w)


def _levels(s_bits, cb_row):
    s = np.uint16(s_bits).view(np.float16)
    return np.array([float(np.float16(s * np.float16(c))) for c in cb_row.view(np.float16)])


def test_quantizer_scales_cover_the_group(small_q4x):
    w, q = small_q4x
    wg = w.reshape(-1, 64).astype(np.float64)
    s = q.scales.reshape(-1).view(np.float16).astype(np.float64)
    amax = np.abs(wg).max(axis=1)
    assert np.all(amax <= s)
    below = (q.scales.reshape(-1) - 1).view(np.float16).astype(np.float64)  # next binary16 down
    assert np.all(below < amax)


def test_quantizer_codes_and_selectors_by_brute_force(small_q4x):
    w, q = small_q4x
    wg = w.reshape(-1, 64).astype(np.float64)
    sel = q.selectors.reshape(-1)
    codes = q.codes.reshape(-1, 64)
    for g in range(wg.shape[0]):
        errs = []
        for t in range(4):
            lv = _levels(q.scales.reshape(-1)[g], q.codebook[t])
            d = np.abs(wg[g][:, None] - lv[None, :])
            errs.append(float((d.min(axis=1) ** 2).sum()))
            if t == sel[g]:
                for i in range(64):
                    best = min(range(16), key=lambda e: (d[i, e], e))
                    assert codes[g, i] == best
        assert sel[g] == min(range(4), key=lambda t: (errs[t], t))


def test_quantizer_codebook_shape_and_order(small_q4x):
    _, q = small_q4x
    cb = q.codebook.view(np.float16).astype(np.float64)
    assert cb.shape == (4, 16)
    assert np.all(np.diff(cb, axis=1) >= 0)
    assert np.all(np.abs(cb) <= 1.0)


def test_reduction_is_a_lloyd_max_fixed_point():
    """Each reduced value is the mean of the learned density over its cell (cells bounded by
    the midpoints of neighbouring values), computed here by direct integration."""
    rng = np.random.default_rng(11)
    pmf = rng.random(32) ** 3
    pmf /= pmf.sum()
    c = qq.reduce_histogram(pmf, max_iter=2000)
    edges = np.linspace(-1, 1, 33)
    bounds = np.concatenate([[-1.0], (c[:-1] + c[1:]) / 2, [1.0]])
    for e in range(16):
        xs = np.linspace(bounds[e], bounds[e + 1], 20001)
        dens = pmf[np.clip(np.searchsorted(edges, xs, side="right") - 1, 0, 31)] / (2 / 32)
        mass = np.trapezoid(dens, xs)
        if mass > 0:
            assert abs(np.trapezoid(dens * xs, xs) / mass - c[e]) < 2e-4


def test_native_assignment_equals_numpy_brute_force():
    w = qi.weights("laplace", 0.008, 4, 10, 16, 1024)
    q = qq.quantize_q4x(w)
    c2, s2 = qq.assign_codes_numpy(w.reshape(-1, 64).astype(np.float64), q.scales.reshape(-1), q.codebook)
    assert np.array_equal(c2, q.codes.reshape(-1, 64))
    assert np.array_equal(s2, q.selectors.reshape(-1))


def test_q4x_beats_rtn_4bit_on_heavy_tailed_weights():
    """The paper's Table 2 ranks Q4X above the 4-bit round-to-nearest format; on the
    heavy-tailed synthetic MLP weights its Frobenius error is below uniform-4 g64."""
    w = qi.weights("t4", 0.0141421, 4, 12, 64, 2048)
    q = qq.quantize_q4x(w)
    wq = q4x.dequant(q.codes, q.scales, q.selectors, q.codebook).astype(np.float64)
    u = qi.quantize_uniform(w, 4, 64)
    wu = oracle.dequant(u.codes, 64, 0, u.scales, u.zeros).astype(np.float64)
    assert np.linalg.norm(wq - w) < np.linalg.norm(wu - w)
