"""Pins of the oracle (CPU only): hand-derived layout examples, identities,
closed forms, exhaustive rounding checks, brute force and the paper's BPW."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
import qx_inputs as qi
import qx_inputs.configs  # noqa: F401  (qi.configs)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ layout
def test_bit_positions_are_a_permutation():
    for bits in (3, 4):
        pos = oracle.chunk_bit_positions(bits)
        assert sorted(pos.ravel().tolist()) == list(range(128 * bits))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("ex", _load("layout_examples.json")["examples"], ids=lambda e: e["name"])
def test_layout_worked_examples(ex):
    n, k, bits = ex["n"], ex["k"], ex["bits"]
    codes = np.zeros((n, k), np.uint8)
    for r, c, v in ex["set"]:
        codes[r, c] = v
    G = k // 128
    blob = oracle.pack(codes, bits, 128, 0, scales=np.zeros((n, G), np.uint16),
                       zeros=np.zeros((n, G), np.uint16))
    code_region = blob[:ex["code_bytes"]]
    want = np.zeros(ex["code_bytes"], np.uint8)
    for off, val in ex["nonzero"].items():
        want[int(off)] = val
    assert np.array_equal(code_region, want)
    back = oracle.unpack(blob, n, k, bits, 128, 0)[0]
    assert np.array_equal(back, codes)


@pytest.mark.parametrize("bits,kind,group", [(3, 0, 64), (3, 1, 128), (4, 0, 128), (4, 1, 64),
                                             (3, 0, 32), (4, 0, 256)])
@pytest.mark.parametrize("n,k", [(1, 128), (3, 256), (5, 384), (2, 1024)])
def test_pack_unpack_identity(bits, kind, group, n, k):
    if k % group:
        pytest.skip("k not a multiple of the group")
    rng = np.random.default_rng(n * k + bits)
    G = k // group
    codes = rng.integers(0, 2**bits, (n, k), dtype=np.uint8)
    if kind == 0:
        s = rng.integers(0, 0x7C00, (n, G), dtype=np.uint16)
        z = np.float16(rng.integers(0, 2**bits, (n, G))).view(np.uint16)
        blob = oracle.pack(codes, bits, group, kind, scales=s, zeros=z)
        c2, s2, z2, _ = oracle.unpack(blob, n, k, bits, group, kind)
        assert np.array_equal(s2, s) and np.array_equal(z2, z)
    else:
        cb = rng.integers(0, 2**16, (n, G, 2**bits), dtype=np.uint16)
        blob = oracle.pack(codes, bits, group, kind, codebook=cb)
        c2, _, _, cb2 = oracle.unpack(blob, n, k, bits, group, kind)
        assert np.array_equal(cb2, cb)
    assert np.array_equal(c2, codes)
    assert blob.size == oracle.packed_size(n, k, bits, group, kind)


@pytest.mark.parametrize("bits", [3, 4])
def test_every_code_position_and_value_alone(bits):
    """Each (position, value) lands on exactly its own bits and unpacks back alone."""
    k = 256
    for pos, val in itertools.product(range(k), range(1, 2**bits)):
        if (pos + val) % 3:  # a third of the (position, value) pairs, covering every position
            continue
        codes = np.zeros((1, k), np.uint8)
        codes[0, pos] = val
        blob = oracle.pack(codes, bits, 128, 1, codebook=np.zeros((1, 2, 2**bits), np.uint16))
        nbits = int(np.unpackbits(blob[:k * bits // 8]).sum())
        assert nbits == bin(val).count("1")
        assert np.array_equal(oracle.unpack(blob, 1, k, bits, 128, 1)[0], codes)


def test_pack_rejects_out_of_range_codes():
    with pytest.raises(ValueError):
        oracle.pack(np.full((1, 128), 8, np.uint8), 3, 128, 1, codebook=np.zeros((1, 1, 8), np.uint16))


# ------------------------------------------------------------------ dequant
def test_dequant_closed_form_small_example():
    s = np.float16([[0.5]]).view(np.uint16)
    z = np.float16([[3.0]]).view(np.uint16)
    codes = np.zeros((1, 128), np.uint8)
    codes[0, :8] = np.arange(8)
    w = oracle.dequant(codes, 128, 0, s, z)
    assert w[0, :8].tolist() == [-1.5, -1.0, -0.5, 0.0, 0.5, 1.0, 1.5, 2.0]
    assert np.all(w[0, 8:] == -1.5)


def test_fp16_product_rounding_is_a_single_rounding_exhaustive():
    """For every finite binary16 s and integer d in [-15, 15], s*d is exact in fp32 and fp64,
    so the fp64 route of the oracle and an fp32 route round the same value once."""
    s = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16)
    s = np.concatenate([s, -s])
    d = np.arange(-15, 16)
    p64 = (s.astype(np.float64)[:, None] * d[None, :])
    p32 = (s.astype(np.float32)[:, None] * d[None, :].astype(np.float32))
    assert np.array_equal(p64, p32.astype(np.float64))
    assert np.array_equal(p64.astype(np.float16).view(np.uint16), p32.astype(np.float16).view(np.uint16))


def test_dequant_codebook_lookup_by_hand():
    cb = np.float16([[[-3, -1, -0.5, 0, 0.25, 1, 2, 7.5]]]).view(np.uint16)
    codes = np.tile(np.arange(8, dtype=np.uint8), 16)[None, :]
    w = oracle.dequant(codes, 128, 1, codebook=cb)
    assert w[0, :8].tolist() == [-3, -1, -0.5, 0, 0.25, 1, 2, 7.5]


def test_dequant_packed_equals_dequant():
    spec = qi.configs.c3()[0]
    q = qi.quantize_codebook(spec.weights(0, 8), 3, 128)
    blob = oracle.pack(q.codes, 3, 128, 1, codebook=q.codebook)
    a = oracle.dequant_packed(blob, 8, spec.k, 3, 128, 1)
    b = oracle.dequant(q.codes, 128, 1, codebook=q.codebook)
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


# ------------------------------------------------------------------ products
def test_gemv_one_hot_gives_column_and_matches_brute_force():
    rng = np.random.default_rng(3)
    w16 = rng.standard_normal((6, 128)).astype(np.float16)
    for j in (0, 5, 127):
        x = np.zeros(128, np.float16)
        x[j] = 1
        assert np.array_equal(oracle.gemv(w16, x), w16[:, j].astype(np.float64))
    x = rng.standard_normal(128).astype(np.float16)
    brute = [sum(float(w16[r, c]) * float(x[c]) for c in range(128)) for r in range(6)]
    assert np.allclose(oracle.gemv(w16, x), brute, rtol=1e-13, atol=1e-13)
    assert np.all(oracle.gemv(w16, np.zeros(128, np.float16)) == 0)


def test_gemm_rows_are_gemv():
    rng = np.random.default_rng(4)
    w16 = rng.standard_normal((10, 256)).astype(np.float16)
    X = rng.standard_normal((3, 256)).astype(np.float16)
    Y = oracle.gemm(X, w16)
    for m in range(3):
        assert np.allclose(Y[m], oracle.gemv(w16, X[m]), rtol=1e-14, atol=1e-14)


def test_normwise_metric():
    assert oracle.normwise_rel_err([1.0, 2.0], [1.0, 2.0]) == 0.0
    assert oracle.normwise_rel_err([1.0, 2.002], [1.0, 2.0]) == pytest.approx(1e-3)
    assert oracle.normwise_rel_err([0.0], [0.0]) == 0.0


# ------------------------------------------------------------------ sizes
def test_paper_bits_per_weight():
    for f in _load("paper_bpw.json")["formats"]:
        if "block_bytes" in f:
            bpw = f["block_bytes"] * 8 / f["block_weights"]
        else:
            bpw = oracle.bits_per_weight(f["bits"], f["group"], f["meta_bits_per_group"])
        assert round(bpw, 2) == f["printed_bpw"], f["name"]


def test_our_formats_bits_per_weight():
    # uniform: fp16 scale + fp16 zero per group; codebook: 2^b fp16 entries per group
    for (n, k, b, g, kind), want in [((4096, 4096, 4, 128, 0), 4.25), ((11008, 4096, 3, 64, 0), 3.5),
                                     ((4096, 4096, 3, 128, 1), 4.0)]:
        assert oracle.packed_size(n, k, b, g, kind) * 8 / (n * k) == want


def test_metadata_bytes_by_hand():
    """Uniform word = scale bits | zero bits << 16, little-endian; codebook entries in order."""
    codes = np.zeros((1, 128), np.uint8)
    s = np.float16([[0.5]]).view(np.uint16)     # 0x3800
    z = np.float16([[3.0]]).view(np.uint16)     # 0x4200
    blob = oracle.pack(codes, 4, 128, 0, scales=s, zeros=z)
    assert blob[64:].tolist() == [0x00, 0x38, 0x00, 0x42]
    cb = np.float16([[[1.0, -2.0, 0, 0, 0, 0, 0, 0]]]).view(np.uint16)  # 0x3C00, 0xC000
    blob = oracle.pack(codes[:, :128], 3, 128, 1, codebook=cb)
    assert blob[48:52].tolist() == [0x00, 0x3C, 0x00, 0xC0] and not blob[52:].any()


def test_dequant_group_index_by_hand():
    """Groups run along k: with g = 64, columns 64j..64j+63 use table j."""
    codes = np.ones((2, 256), np.uint8)
    s = np.float16([[1, 2, 4, 8], [0.5, 0.25, 0.125, 3]]).view(np.uint16)
    z = np.zeros((2, 4), np.uint16)
    w = oracle.dequant(codes, 64, 0, s, z)
    assert np.array_equal(w[:, ::64], np.float16([[1, 2, 4, 8], [0.5, 0.25, 0.125, 3]]))
    assert np.all(w.reshape(2, 4, 64) == w.reshape(2, 4, 64)[:, :, :1])
    cb = np.zeros((2, 4, 8), np.float16)
    cb[:, :, 1] = [[1, 2, 4, 8], [5, 6, 7, 9]]
    w = oracle.dequant(codes, 64, 1, codebook=cb.view(np.uint16))
    assert np.array_equal(w[:, ::64], cb[:, :, 1])
