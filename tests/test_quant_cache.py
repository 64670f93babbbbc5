"""The disk cache of quantized synthetic matrices (input preparation, CPU only)."""
import numpy as np
import pytest

from qx_inputs import cache, configs


@pytest.fixture
def cache_env(tmp_path, monkeypatch):
    monkeypatch.setenv("QX_QUANT_CACHE", str(tmp_path / "qc"))
    monkeypatch.setenv("QX_QUANT_CACHE_GB", "1")
    return tmp_path / "qc"


def _same(a, b):
    for f in ("codes", "scales", "zeros", "codebook", "selectors"):
        x, y = getattr(a, f), getattr(b, f)
        assert (x is None) == (y is None), f
        if x is not None:
            assert x.dtype == y.dtype and np.array_equal(x, y), f


@pytest.mark.parametrize("kind", [configs.UNIFORM, configs.CODEBOOK, configs.Q4X])
def test_cached_matrix_equals_fresh_quantization(cache_env, monkeypatch, kind):
    bits, g = (4, 64) if kind == configs.Q4X else (3, 128 if kind == configs.CODEBOOK else 64)
    spec = configs.MatrixSpec("t", 40, 512, "t4", 0.02, 9, 1, bits, g, kind)
    first = spec.quantized(3, 17)                 # quantized and stored
    assert cache.load(spec, 3, 17) is not None
    second = spec.quantized(3, 17)                # read back
    _same(first, second)
    assert second.meta["spec"] == spec and second.meta["row0"] == 3
    monkeypatch.setenv("QX_QUANT_CACHE", "off")
    _same(first, spec.quantized(3, 17))           # and equal to a fresh quantization


def test_key_covers_the_spec_and_rows(cache_env):
    a = configs.MatrixSpec("t", 40, 512, "t4", 0.02, 9, 1, 3, 64, configs.UNIFORM)
    keys = {cache.key(a, 0, None), cache.key(a, 0, 8), cache.key(a, 1, 8),
            cache.key(configs.MatrixSpec("t", 40, 512, "t4", 0.02, 9, 2, 3, 64, configs.UNIFORM), 0, None),
            cache.key(configs.MatrixSpec("t", 40, 512, "t4", 0.02, 9, 1, 4, 64, configs.UNIFORM), 0, None)}
    assert len(keys) == 5


def test_budget_and_off(cache_env, monkeypatch):
    spec = configs.MatrixSpec("t", 64, 1024, "normal", 0.02, 4, 0, 4, 128, configs.UNIFORM)
    monkeypatch.setenv("QX_QUANT_CACHE_GB", "0.00001")  # 10 kB: the 64 kB of codes do not fit
    spec.quantized()
    assert cache.load(spec, 0, None) is None
    monkeypatch.setenv("QX_QUANT_CACHE", "off")
    assert cache.cache_dir() is None and not cache.store(spec, 0, None, spec.quantized())
