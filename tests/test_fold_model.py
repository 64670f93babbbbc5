"""CPU model of the fp32 summation order of the uniform-group GEMV (no GPU).

The uniform GEMV kernels feed codes to the fp16 dot products as "M + q" (the
code in the fraction bits of a binary16 whose exponent makes one fraction step
worth 1), and take the bias out once per group: a group contributes
s * (sum (M+q)x - sum Mx - z sum x), which is s * sum (q-z)x in exact
arithmetic (the uniform levels of Section 2.2, W' = s(q - z)).

In fp32 the two large sums are rounded, so their difference carries a residual
of the size of u * M * sum|x|, multiplied by s. The quantizer stores s = 1 for a
group whose weights are all zero, so with two *different* summation orders the
residual of such a group lands in y unscaled. The kernels therefore form both
sums with the same instructions in the same order: every 8-code piece is summed
by its own 4-step dot2 chain, and the pieces of a group are added in the
balanced pairwise order of the DPP reduction that stages sum Mx. A zero group
then gives exactly 0, and every other group's residual is proportional to s.

The model below reproduces both orders for 4-bit codes in groups of 128 and
3-bit codes in groups of 64 (v_dot2_f32_f16 taken as the fp32 rounding of the
exact a0*b0 + a1*b1 + c, which is what the instruction returns for normal fp16
inputs within one fp32 ulp).
"""
import numpy as np
import pytest

U32 = np.float32


def dot2(a0, a1, b0, b1, c):
    """fp32 rounding of a0*b0 + a1*b1 + c (fp16 a, b; fp32 c), vectorised over trials."""
    return (np.float64(a0) * b0 + np.float64(a1) * b1 + np.float64(c)).astype(U32)


def tree(parts):
    """Balanced pairwise sum in fp32, the order of the lane reductions (xor 1, xor 2, mirrors)."""
    parts = list(parts)
    while len(parts) > 1:
        parts = [(parts[i] + parts[i + 1]).astype(U32) for i in range(0, len(parts), 2)]
    return parts[0]


def u4_slots(x8, q8):
    """Decoder pair order of one 8-value piece of a 4-bit chunk: (0,4) (1,5) (2,6) (3,7),
    with the bias of each slot (bits 0-3 of a half: M = 1024, bits 4-7: M = 64)."""
    return [((0, 4), 1024.0), ((1, 5), 64.0), ((2, 6), 1024.0), ((3, 7), 64.0)]


def u4g128_group(x, q, s, z, order):
    """One group of 128 codes (x: [T, 128] fp16 values as float64, q: [128] codes)."""
    T = x.shape[0]
    zero = np.zeros(T, U32)
    pieces = [(x[:, 8 * p:8 * p + 8], q[8 * p:8 * p + 8]) for p in range(16)]
    sx = tree([_chain([(xp[:, 2 * i], xp[:, 2 * i + 1], 1.0, 1.0) for i in range(4)], zero)
               for xp, _ in pieces])
    if order == "biased_fold_separate_orders":
        # staging: natural-order pairs (x0,x1)..(x6,x7) against (1024, 64); chunk: one chain
        mx = tree([_chain([(xp[:, 2 * i], xp[:, 2 * i + 1], 1024.0, 64.0) for i in range(4)], zero)
                   for xp, _ in pieces])
        acc = zero
        for xp, qp in pieces:
            for (i, j), M in u4_slots(xp, qp):
                acc = dot2(M + qp[i], M + qp[j], xp[:, i], xp[:, j], acc)
    else:  # per-piece chains in decoder order, the same balanced tree on both sides
        mx = tree([_chain([(xp[:, i], xp[:, j], M, M) for (i, j), M in u4_slots(xp, qp)], zero)
                   for xp, qp in pieces])
        acc = tree([_chain([(xp[:, i], xp[:, j], M + qp[i], M + qp[j]) for (i, j), M in u4_slots(xp, qp)],
                           zero) for xp, qp in pieces])
    t = ((np.float64(acc - mx) - np.float64(z) * sx)).astype(U32)  # fma(-z, sx, acc - mx)
    return (U32(s) * t).astype(U32)


def u3g64_groups(x, q, s, z, order):
    """The two groups of 64 of one 3-bit chunk. Codes 0-47 sit in bits 0-2 (M = 1024),
    48-95 in bits 3-5 (M = 128), 96-127 in the spare fields (M = 16); decoder pairs per
    4 codes are (0,2) (1,3). Group 0 = pieces 0-7, group 1 = pieces 8-15."""
    T = x.shape[0]
    zero = np.zeros(T, U32)
    M_of = lambda p: 1024.0 if p < 6 else 128.0 if p < 12 else 16.0
    slots = [(0, 2), (1, 3), (4, 6), (5, 7)]
    out = []
    for g in range(2):
        ps = range(8 * g, 8 * g + 8)
        sx = tree([_chain([(x[:, 8 * p + 2 * i], x[:, 8 * p + 2 * i + 1], 1.0, 1.0) for i in range(4)], zero)
                   for p in ps])
        if order == "biased_fold_separate_orders":
            # staging: M * (sum x of the piece); chunk: one chain per group, fed code dword
            # by code dword (dword i: the 4-code block of bits 0-2 at codes 4i.., then that of
            # bits 3-5 at 48 + 4i..; then the spare codes 96 + 4i.. of dwords 0-7)
            mx = tree([(U32(M_of(p)) * _chain([(x[:, 8 * p + 2 * i], x[:, 8 * p + 2 * i + 1], 1.0, 1.0)
                                               for i in range(4)], zero)).astype(U32) for p in ps])
            acc = zero
            starts = [c for i in range(12) for c in (4 * i, 48 + 4 * i)] + [96 + 4 * i for i in range(8)]
            for c0 in starts:
                if c0 // 64 != g:
                    continue
                M = M_of(c0 // 8)
                for i, j in ((0, 2), (1, 3)):
                    acc = dot2(M + q[c0 + i], M + q[c0 + j], x[:, c0 + i], x[:, c0 + j], acc)
        else:
            mx = tree([_chain([(x[:, 8 * p + i], x[:, 8 * p + j], M_of(p), M_of(p)) for i, j in slots], zero)
                       for p in ps])
            acc = tree([_chain([(x[:, 8 * p + i], x[:, 8 * p + j], M_of(p) + q[8 * p + i], M_of(p) + q[8 * p + j])
                                for i, j in slots], zero) for p in ps])
        t = ((np.float64(acc - mx) - np.float64(z[g]) * sx)).astype(U32)
        out.append((U32(s[g]) * t).astype(U32))
    return out


def _chain(terms, c):
    for b0, b1, a0, a1 in terms:
        c = dot2(a0, a1, b0, b1, c)
    return c


def _x(T, n, seed, outliers=False):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, n))
    if outliers:  # about 1 % of the channels x20, as in the outlier-activation workload
        for t in range(T):
            x[t, rng.choice(n, max(1, n // 100), replace=False)] *= 20
    return x.astype(np.float16).astype(np.float64)


@pytest.mark.parametrize("outliers", [False, True])
def test_zero_group_residual(outliers):
    """All-zero group (s = 1, z = 0, q = 0): the separate orders leave a residual of
    order 1e-3 in y; the shared order gives exactly zero."""
    T = 200
    x = _x(T, 128, seed=11 + outliers, outliers=outliers)
    q = np.zeros(128, np.int64)
    old = u4g128_group(x, q, 1.0, 0.0, "biased_fold_separate_orders")
    new = u4g128_group(x, q, 1.0, 0.0, "shared")
    assert np.max(np.abs(old)) > 1e-4  # the defect the shared order removes
    assert np.all(new == 0)
    x3 = _x(T, 128, seed=21 + outliers, outliers=outliers)
    q3 = np.zeros(128, np.int64)
    old3 = u3g64_groups(x3, q3, [1.0, 1.0], [0.0, 0.0], "biased_fold_separate_orders")
    new3 = u3g64_groups(x3, q3, [1.0, 1.0], [0.0, 0.0], "shared")
    assert max(np.max(np.abs(v)) for v in old3) > 1e-5
    assert all(np.all(v == 0) for v in new3)
    print(f"zero group, outliers={outliers}: separate orders max|y| 4-bit {np.max(np.abs(old)):.2e}, "
          f"3-bit {max(np.max(np.abs(v)) for v in old3):.2e}; shared order 0")


@pytest.mark.parametrize("outliers", [False, True])
def test_shared_order_residual_scales_with_levels(outliers):
    """Non-degenerate groups: the error of the shared order against the exact
    s * sum (q - z) x stays within u * s * (M + 2^b) * sum|x| times a small count
    of roundings, i.e. it scales with the group's scale s."""
    T, rng = 200, np.random.default_rng(5)
    x = _x(T, 128, seed=31 + outliers, outliers=outliers)
    u = 2.0 ** -24
    for s in (2.0 ** -9, 1.0, 2.0 ** 6):
        q = rng.integers(0, 16, 128)
        z = float(rng.integers(0, 16))
        y = u4g128_group(x, q, s, z, "shared").astype(np.float64)
        exact = s * (x @ (q - z))
        bound = 12 * u * s * (1024 + 16) * np.abs(x).sum(axis=1)
        assert np.all(np.abs(y - exact) <= bound)
        q3 = rng.integers(0, 8, 128)
        z3 = [float(rng.integers(0, 8)), float(rng.integers(0, 8))]
        y3 = u3g64_groups(x, q3, [s, s], z3, "shared")
        for g in range(2):
            ex3 = s * (x[:, 64 * g:64 * g + 64] @ (q3[64 * g:64 * g + 64] - z3[g]))
            b3 = 12 * u * s * (1024 + 8) * np.abs(x[:, 64 * g:64 * g + 64]).sum(axis=1)
            assert np.all(np.abs(y3[g].astype(np.float64) - ex3) <= b3)
