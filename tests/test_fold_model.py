"""CPU model of the fp32 arithmetic of the uniform-group GEMV (no GPU).

A uniform group contributes s * sum (q - z) x to y (the uniform levels of
Section 2.2, W' = s(q - z)). The GEMV kernels feed each code to the fp16 dot
products as the masked code field alone, which reads as a binary16 subnormal
q * 2^(f - 24) (f the field's lowest bit in its half), keep one fp32 accumulator
per field kind, and fold the zero point once per group:

    y_g = s * fma(-z, sum x, 2^24 f_0 + 2^20 f_1)          (b = 4)
    y_g = s * fma(-z, sum x, 2^24 f_0 + 2^21 f_1 + 2^18 f_2) (b = 3)

No bias enters the sums, so a group whose codes are all 0 gives exactly 0 (the
quantizer stores an all-zero group with s = 1, z = 0), and the rounding error
of both sums is of the size of u * s * (2^b + z) * sum|x|: it scales with the
group's levels. An earlier form fed codes as M + q (M = 1024, 128, 64, 16 by
field) and subtracted a staged sum M x; its residual, u * s * M * sum|x|, did
not vanish for s = 1 unless both sums were rounded in the same order. The model
reproduces the kernel's order for 4-bit codes in groups of 128 and 3-bit codes
in groups of 64 (v_dot2_f32_f16 taken as the fp32 rounding of the exact
a0*b0 + a1*b1 + c; the instruction returns that within two fp32 ulps, and
keeps subnormal binary16 inputs), next to the old biased form.
"""
import numpy as np
import pytest

U32 = np.float32
U = 2.0 ** -24


def dot2(a0, a1, b0, b1, c):
    """fp32 rounding of a0*b0 + a1*b1 + c (fp16 a, b; fp32 c), vectorised over trials."""
    return (np.float64(a0) * b0 + np.float64(a1) * b1 + np.float64(c)).astype(U32)


def fma32(a, b, c):
    return (np.float64(a) * np.float64(b) + np.float64(c)).astype(U32)


def tree(parts):
    """Balanced pairwise sum in fp32 (the lane reductions of the staged sum x)."""
    parts = list(parts)
    while len(parts) > 1:
        parts = [(parts[i] + parts[i + 1]).astype(U32) for i in range(0, len(parts), 2)]
    return parts[0]


def _sum_x(x, lo, hi):
    """sum x over codes [lo, hi): one (1, 1) dot2 chain per 8-value piece, pieces by tree."""
    zero = np.zeros(x.shape[0], U32)
    parts = []
    for p in range(lo // 8, hi // 8):
        c = zero
        for i in range(4):
            c = dot2(1.0, 1.0, x[:, 8 * p + 2 * i], x[:, 8 * p + 2 * i + 1], c)
        parts.append(c)
    return tree(parts)


def u4g128_group(x, q, s, z, form):
    """One group of 128 4-bit codes (x: [T, 128] fp16 values as float64)."""
    zero = np.zeros(x.shape[0], U32)
    sx = _sum_x(x, 0, 128)
    if form == "raw":
        f = [zero, zero]  # bits 0-3 (unit 2^-24), bits 4-7 (unit 2^-20)
        for j in range(16):  # code dword j: pairs (0,4) (1,5) (2,6) (3,7) of codes 8j..
            for (a, b), kind in (((0, 4), 0), ((1, 5), 1), ((2, 6), 0), ((3, 7), 1)):
                unit = 2.0 ** -24 if kind == 0 else 2.0 ** -20
                f[kind] = dot2(q[8 * j + a] * unit, q[8 * j + b] * unit, x[:, 8 * j + a], x[:, 8 * j + b],
                               f[kind])
        A = fma32(f[1], 2.0 ** 20, (f[0] * U32(2.0 ** 24)).astype(U32))
        return (U32(s) * fma32(-z, sx, A)).astype(U32)
    # biased form, summed in two different orders (staging: natural pairs; chunk: one chain)
    mx = zero
    parts = []
    for p in range(16):
        c = zero
        for i in range(4):
            c = dot2(1024.0, 64.0, x[:, 8 * p + 2 * i], x[:, 8 * p + 2 * i + 1], c)
        parts.append(c)
    mx = tree(parts)
    acc = zero
    for j in range(16):
        for (a, b), M in (((0, 4), 1024.0), ((1, 5), 64.0), ((2, 6), 1024.0), ((3, 7), 64.0)):
            acc = dot2(M + q[8 * j + a], M + q[8 * j + b], x[:, 8 * j + a], x[:, 8 * j + b], acc)
    t = (np.float64((acc - mx).astype(U32)) - np.float64(z) * sx).astype(U32)
    return (U32(s) * t).astype(U32)


def u3g64_groups(x, q, s, z):
    """The two groups of 64 of one 3-bit chunk, raw form. Codes 0-47 sit in bits 0-2
    (unit 2^-24), 48-95 in bits 3-5 (2^-21), 96-127 in the spare fields, bits 6-8
    (2^-18); decoder pairs per 4 codes are (0,2) (1,3); code dword i feeds codes 4i..
    (bits 0-2) and 48+4i.. (bits 3-5), spare dword i codes 96+4i.."""
    zero = np.zeros(x.shape[0], U32)
    f = [[zero, zero, zero] for _ in range(2)]
    units = [2.0 ** -24, 2.0 ** -21, 2.0 ** -18]
    blocks = [(4 * i, 0) for i in range(12)] + [(48 + 4 * i, 1) for i in range(12)]
    order = []
    for i in range(0, 12, 2):  # the kernel's loop: dwords i, i+1, fields a then b
        for h in range(2):
            order += [(4 * (i + h), 0), (48 + 4 * (i + h), 1)]
    order += [(96 + 4 * i, 2) for i in range(8)]
    assert sorted(order) == sorted(blocks + [(96 + 4 * i, 2) for i in range(8)])
    for c0, kind in order:
        g = c0 // 64
        for a, b in ((0, 2), (1, 3)):
            f[g][kind] = dot2(q[c0 + a] * units[kind], q[c0 + b] * units[kind], x[:, c0 + a], x[:, c0 + b],
                              f[g][kind])
    out = []
    for g in range(2):
        A = fma32(f[g][2], 2.0 ** 18, fma32(f[g][1], 2.0 ** 21, (f[g][0] * U32(2.0 ** 24)).astype(U32)))
        out.append((U32(s[g]) * fma32(-z[g], _sum_x(x, 64 * g, 64 * g + 64), A)).astype(U32))
    return out


def _x(T, n, seed, outliers=False):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, n))
    if outliers:  # about 1 % of the channels x20, as in the outlier-activation workload
        for t in range(T):
            x[t, rng.choice(n, max(1, n // 100), replace=False)] *= 20
    return x.astype(np.float16).astype(np.float64)


def test_subnormal_codes_are_exact():
    """Every code of every field kind, placed in its bits, is the binary16 value q times
    the field's unit (a subnormal), which is what the model multiplies."""
    for bits, shifts in ((4, (0, 4)), (3, (0, 3, 6))):
        for sh in shifts:
            for q in range(1 << bits):
                h = np.array([q << sh], np.uint16).view(np.float16)[0]
                assert float(h) == q * 2.0 ** (sh - 24)


@pytest.mark.parametrize("outliers", [False, True])
def test_zero_group_is_exactly_zero(outliers):
    """All-zero group (s = 1, z = 0, q = 0): exactly 0 in the kernel's arithmetic; the
    old biased form, summed in two orders, left a residual of order 1e-3."""
    T = 200
    x = _x(T, 128, seed=11 + outliers, outliers=outliers)
    q = np.zeros(128, np.int64)
    raw = u4g128_group(x, q, 1.0, 0.0, "raw")
    old = u4g128_group(x, q, 1.0, 0.0, "biased")
    assert np.all(raw == 0)
    assert np.max(np.abs(old)) > 1e-4
    raw3 = u3g64_groups(_x(T, 128, seed=21 + outliers, outliers=outliers), q, [1.0, 1.0], [0.0, 0.0])
    assert all(np.all(v == 0) for v in raw3)
    print(f"zero group, outliers={outliers}: raw 0, old biased form max|y| {np.max(np.abs(old)):.2e}")


@pytest.mark.parametrize("outliers", [False, True])
def test_error_scales_with_levels(outliers):
    """Non-degenerate groups: against the exact s * sum (q - z) x the error stays within
    n_roundings * u * s * (2^b - 1 + z) * sum|x| (plus one rounding of the result): it
    scales with s, and it is far below the old biased form's."""
    T, rng = 200, np.random.default_rng(5)
    x = _x(T, 128, seed=31 + outliers, outliers=outliers)
    worst_raw = worst_old = 0.0
    for s in (2.0 ** -9, 1.0, 2.0 ** 6):
        q = rng.integers(0, 16, 128)
        z = float(rng.integers(0, 16))
        exact = s * (x @ (q - z))
        ax = np.abs(x).sum(axis=1)
        y = u4g128_group(x, q, s, z, "raw").astype(np.float64)
        bound = 70 * U * s * (15 + z) * ax + U * np.abs(exact)
        assert np.all(np.abs(y - exact) <= bound)
        old = u4g128_group(x, q, s, z, "biased").astype(np.float64)
        worst_raw = max(worst_raw, float(np.max(np.abs(y - exact) / (s * ax))))
        worst_old = max(worst_old, float(np.max(np.abs(old - exact) / (s * ax))))
        q3 = rng.integers(0, 8, 128)
        z3 = [float(rng.integers(0, 8)), float(rng.integers(0, 8))]
        y3 = u3g64_groups(x, q3, [s, s], z3)
        for g in range(2):
            xs = x[:, 64 * g:64 * g + 64]
            ex3 = s * (xs @ (q3[64 * g:64 * g + 64] - z3[g]))
            b3 = 40 * U * s * (7 + z3[g]) * np.abs(xs).sum(axis=1) + U * np.abs(ex3)
            assert np.all(np.abs(y3[g].astype(np.float64) - ex3) <= b3)
    assert worst_raw * 20 < worst_old  # the raw codes are at least 20x tighter than the bias
    print(f"outliers={outliers}: max |err| / (s sum|x|) raw {worst_raw:.2e}, old biased {worst_old:.2e}")
