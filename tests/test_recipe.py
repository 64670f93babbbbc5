"""The offline recipe tool (CPU): reconstruction equals the oracle's dequantization,
the Lagrangian allocation is optimal among allocations using no more bytes (brute
force), fits its budget, and loosening the budget never raises the error."""
import itertools

import numpy as np
import pytest

import oracle
from oracle import q4x
import qx_inputs as qi
from qx_inputs import recipe


@pytest.mark.parametrize("cand", recipe.CANDIDATES, ids=lambda c: c[0])
def test_reconstruction_matches_oracle(cand):
    _, bits, group, kind = cand
    q = qi.quantize(qi.weights("laplace", 0.008, 7, 1, 6, 512), bits, group, kind)
    if kind == qi.Q4X:
        ref = q4x.dequant(q.codes, q.scales, q.selectors, q.codebook)
    else:
        ref = oracle.dequant(q.codes, group, kind, q.scales, q.zeros, q.codebook)
    assert np.array_equal(recipe.reconstruct(q), ref.astype(np.float64))


def test_bits_per_weight_of_the_candidates():
    got = {c: recipe.bits_per_weight(b, g, k) for c, b, g, k in recipe.CANDIDATES}
    assert got["U4g128"] == 4.25 and got["U3g64"] == 3.5 and got["CB3g128"] == 4.0
    assert got["Q4X"] == 4 + 18 / 64


def _random_instance(rng, n_mats):
    mats = []
    for i in range(n_mats):
        base = rng.uniform(0.5, 2.0)
        sq = {c: base * 2.0 ** (-2 * b) * rng.uniform(0.7, 1.3) for c, b, g, k in recipe.CANDIDATES}
        mats.append(recipe.MatrixErrors(f"m{i}", int(rng.integers(1, 5)) * 4096, sq, {}))
    return mats


@pytest.mark.parametrize("seed", range(6))
def test_allocation_is_optimal_for_the_bytes_it_uses(seed):
    rng = np.random.default_rng(seed)
    mats = _random_instance(rng, 4)
    names = [c for c, *_ in recipe.CANDIDATES]
    all_allocs = [dict(zip([m.name for m in mats], combo)) for combo in itertools.product(names, repeat=len(mats))]
    lo = min(recipe.totals(mats, a)[0] for a in all_allocs)
    hi = max(recipe.totals(mats, a)[0] for a in all_allocs)
    for frac in (0.1, 0.35, 0.6, 0.9):
        budget = lo + frac * (hi - lo)
        alloc = recipe.allocate(mats, budget)
        b, e = recipe.totals(mats, alloc)
        assert b <= budget + 1e-6
        better = [a for a in all_allocs if recipe.totals(mats, a)[0] <= b + 1e-9
                  and recipe.totals(mats, a)[1] < e - 1e-12]
        assert not better


def test_looser_budget_never_raises_error():
    mats = _random_instance(np.random.default_rng(9), 12)
    w = sum(m.weights for m in mats)
    errs = [recipe.totals(mats, recipe.allocate(mats, bpw * w / 8))[1] for bpw in (3.5, 3.75, 4.0, 4.25, 4.5)]
    assert all(a >= b - 1e-12 for a, b in zip(errs, errs[1:]))


def test_budget_below_every_format_is_an_error():
    mats = _random_instance(np.random.default_rng(1), 3)
    with pytest.raises(ValueError):
        recipe.allocate(mats, 1.0)


def test_decoder_recipe_small():
    r = recipe.decoder_recipe(4.0, layers=1, rows=32)
    assert r["achieved_bpw"] <= 4.0 + 1e-9
    assert set(r["formats"]) == {f"L0.{m}" for m in ("q", "k", "v", "o", "gate", "up", "down")}
