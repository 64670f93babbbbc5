"""C-ABI checks that need no GPU: the library loads, exports every declared
entry point, packs byte-identically with the oracle, and returns the
documented status codes. No kernel is launched here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import qx_inputs as qi
from qx_inputs import configs
import paper_2505_07531_amd as qx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header, prefix):
    with open(os.path.join(ROOT, "include", header)) as f:
        hdr = f.read()
    return set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(" + prefix + r"\w+)\s*\(", hdr, re.M))


def test_library_exports_every_declared_symbol():
    declared = _declared("qx.h", "qx_")
    assert {"qx_pack_layout", "qx_dequant", "qx_gemv", "qx_gemm", "qx_status_str"} <= declared
    lib = ctypes.CDLL(qx.LIB_PATH if os.path.exists(qx.LIB_PATH) else qx.build())
    for name in sorted(declared):
        assert hasattr(lib, name), name


def test_every_header_is_checked_against_its_library():
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == ["qx.h", "qx_probe.h"]


def test_probe_library_exports_and_rejects_bad_arguments():
    from paper_2505_07531_amd import probe
    declared = _declared("qx_probe.h", "qxp_")
    assert declared == {"qxp_read", "qxp_empty"}
    lib = probe.load()
    for name in sorted(declared):
        assert hasattr(lib, name), name
    # each call fails an argument check, so nothing is launched
    assert lib.qxp_read(None, 16, None, None) == -1
    assert lib.qxp_read(64, 0, 64, None) == -1      # empty read
    assert lib.qxp_read(64, 24, 64, None) == -1     # not a multiple of 16
    assert lib.qxp_read(8, 16, 64, None) == -1      # src not 16-byte aligned
    assert lib.qxp_empty(0, 64, None) == -1
    assert lib.qxp_empty((1 << 20) + 1, 64, None) == -1
    assert lib.qxp_empty(1, None, None) == -1


def _random_quant(n, k, bits, group, kind, seed):
    rng = np.random.default_rng(seed)
    G = k // group
    codes = rng.integers(0, 2**bits, (n, k), dtype=np.uint8)
    if kind == 0:
        s = np.float16(rng.uniform(1e-4, 1, (n, G))).view(np.uint16)
        z = np.float16(rng.integers(0, 2**bits, (n, G))).view(np.uint16)
        return codes, s, z, None
    cb = np.float16(rng.standard_normal((n, G, 2**bits))).view(np.uint16)
    return codes, None, None, cb


@pytest.mark.parametrize("bits", [3, 4])
@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("n,k", [(1, 128), (7, 384), (300, 256), (3, 11008)])
def test_pack_layout_matches_oracle_bytes(bits, kind, group, n, k):
    codes, s, z, cb = _random_quant(n, k, bits, group, kind, n + k + bits)
    d = qx.desc(n, k, bits, group, kind)
    blob = qx.qx_pack_layout(d, codes, s, z, cb)
    ref = oracle.pack(codes, bits, group, kind, scales=s, zeros=z, codebook=cb)
    assert blob.size == ref.size == oracle.packed_size(n, k, bits, group, kind)
    assert np.array_equal(blob, ref)


@pytest.mark.parametrize("make", [configs.c1, configs.c2, configs.c3])
def test_pack_layout_full_config_matches_oracle(make):
    spec, _ = make()
    q = spec.quantized()
    d = qx.desc(q.n, q.k, q.bits, q.group, q.kind)
    blob = qx.qx_pack_layout(d, q.codes, q.scales, q.zeros, q.codebook)
    ref = oracle.pack(q.codes, q.bits, q.group, q.kind, q.scales, q.zeros, q.codebook)
    assert blob.size == spec.packed_bytes
    assert np.array_equal(blob, ref)


def _st(fn):
    try:
        fn()
    except qx.QxError as e:
        return e.status
    return qx.QX_OK


def test_descriptor_errors():
    codes = np.zeros((1, 128), np.uint8)
    s = np.float16([[1.0]]).view(np.uint16)
    z = np.float16([[0.0]]).view(np.uint16)
    good = dict(n=1, k=128, bits=3, group=128, kind=0)
    for change, want in [(dict(bits=2), qx.QX_E_UNSUPPORTED), (dict(bits=8), qx.QX_E_UNSUPPORTED),
                         (dict(bits=0), qx.QX_E_ARG), (dict(bits=9), qx.QX_E_ARG),
                         (dict(k=100), qx.QX_E_ARG), (dict(k=0), qx.QX_E_ARG),
                         (dict(n=-1), qx.QX_E_ARG), (dict(group=0), qx.QX_E_ARG),
                         (dict(group=48), qx.QX_E_ARG), (dict(group=256, k=256), qx.QX_E_UNSUPPORTED),
                         (dict(group=16), qx.QX_E_UNSUPPORTED), (dict(kind=2), qx.QX_E_ARG)]:
        p = {**good, **change}
        d = qx.desc(p["n"], p["k"], p["bits"], p["group"], p["kind"])
        assert _st(lambda: qx.qx_packed_size(d)) == want, change
    d = qx.desc(1, 128, 3, 128, 0, flags=1)
    assert _st(lambda: qx.qx_packed_size(d)) == qx.QX_E_ARG
    d = qx.desc(1, 128, 3, 128, 0)
    assert _st(lambda: qx.qx_pack_layout(d, codes, s, z)) == qx.QX_OK


def test_pack_layout_value_errors_and_capacity():
    d = qx.desc(2, 128, 3, 64, 0)
    codes = np.zeros((2, 128), np.uint8)
    s = np.float16(np.ones((2, 2))).view(np.uint16)
    z = np.float16(np.zeros((2, 2))).view(np.uint16)
    ok = lambda **kw: _st(lambda: qx.qx_pack_layout(d, **{**dict(codes=codes, scales=s, zeros=z), **kw}))
    assert ok() == qx.QX_OK
    assert ok(codes=np.full((2, 128), 8, np.uint8)) == qx.QX_E_ARG           # code >= 2^b
    assert ok(zeros=np.float16(np.full((2, 2), 2.5)).view(np.uint16)) == qx.QX_E_ARG  # not integer
    assert ok(zeros=np.float16(np.full((2, 2), 8.0)).view(np.uint16)) == qx.QX_E_ARG  # > 2^b - 1
    assert ok(zeros=np.float16(np.full((2, 2), -1.0)).view(np.uint16)) == qx.QX_E_ARG
    assert ok(scales=np.float16(np.full((2, 2), np.inf)).view(np.uint16)) == qx.QX_E_ARG
    assert ok(scales=None) == qx.QX_E_ARG
    assert qx.qx_packed_size(d) == 2 * 128 * 3 // 8 + 2 * 2 * 4
    small = np.empty(qx.qx_packed_size(d) - 1, np.uint8)
    assert _st(lambda: qx.qx_pack_layout(d, codes, s, z, out=small)) == qx.QX_E_SIZE
    dc = qx.desc(2, 128, 3, 64, 1)
    assert _st(lambda: qx.qx_pack_layout(dc, codes)) == qx.QX_E_ARG             # no codebook
    cb = np.full((2, 2, 8), 0x7E00, np.uint16)                                 # NaN entries allowed
    assert _st(lambda: qx.qx_pack_layout(dc, codes, codebook=cb)) == qx.QX_OK


def test_empty_matrix():
    d = qx.desc(0, 256, 4, 128, 0)
    assert qx.qx_packed_size(d) == 0
    assert qx.qx_pack_layout(d, np.zeros((0, 256), np.uint8), np.zeros((0, 2), np.uint16),
                             np.zeros((0, 2), np.uint16)).size == 0


def test_device_calls_reject_bad_arguments_before_launch():
    lib = qx.load()
    d = qx.desc(4, 128, 4, 128, 0)
    P = ctypes.c_void_p
    assert lib.qx_gemv(ctypes.byref(d), None, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemv(ctypes.byref(d), P(16), P(24), P(16), None) == qx.QX_E_ARG   # x misaligned
    assert lib.qx_gemv(ctypes.byref(d), P(16), P(16), P(17), None) == qx.QX_E_ARG   # y odd address
    assert lib.qx_dequant(ctypes.byref(d), P(16), 7, P(16), None) == qx.QX_E_ARG    # bad out_kind
    assert lib.qx_dequant(ctypes.byref(d), P(8), 0, P(16), None) == qx.QX_E_ARG     # misaligned blob
    assert lib.qx_gemm(ctypes.byref(d), P(16), -1, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemm(ctypes.byref(d), P(16), 70000, P(16), P(16), None) == qx.QX_E_ARG
    bad = qx.desc(4, 128, 2, 128, 0)
    assert lib.qx_gemv(ctypes.byref(bad), P(16), P(16), P(16), None) == qx.QX_E_UNSUPPORTED
    assert lib.qx_gemv(None, P(16), P(16), P(16), None) == qx.QX_E_ARG
    # empty work is a no-op that never reaches the runtime
    z = qx.desc(0, 128, 4, 128, 0)
    assert lib.qx_gemv(ctypes.byref(z), None, None, None, None) == qx.QX_OK
    assert lib.qx_gemm(ctypes.byref(d), None, 0, None, None, None) == qx.QX_OK
    assert lib.qx_dequant(ctypes.byref(z), None, 0, None, None) == qx.QX_OK


def test_status_strings():
    assert qx.qx_status_str(0) == "ok"
    assert qx.qx_status_str(-3) == "output buffer too small"
    assert qx.qx_status_str(99) == "unknown status"


# ------------------------------------------------------------------ Q4X (host side)
def _random_q4x(n, k, seed):
    rng = np.random.default_rng(seed)
    G = k // 64
    return (rng.integers(0, 16, (n, k), dtype=np.uint8), rng.integers(0, 2**16, (n, G), dtype=np.uint16),
            rng.integers(0, 4, (n, G), dtype=np.uint8), rng.integers(0, 2**16, (4, 16), dtype=np.uint16))


@pytest.mark.parametrize("n,k", [(1, 128), (3, 1152), (5, 11008), (17, 4096), (2, 16384)])
def test_pack_q4x_matches_oracle_bytes(n, k):
    codes, s, sel, cb = _random_q4x(n, k, n * 31 + k)
    blob = qx.qx_pack_q4x(qx.desc(n, k, 4, 64, qx.QX_Q4X), codes, s, sel, cb)
    assert np.array_equal(blob, oracle.q4x.pack(codes, s, sel, cb))


def test_pack_q4x_quantized_matrix_matches_oracle_bytes():
    from qx_inputs import q4x as qq
    q = qq.quantize_q4x(qi.weights("t4", 0.0141421, 4, 3, 40, 1152))
    blob = qx.qx_pack_q4x(qx.desc(40, 1152, 4, 64, qx.QX_Q4X), q.codes, q.scales, q.selectors, q.codebook)
    assert np.array_equal(blob, oracle.q4x.pack(q.codes, q.scales, q.selectors, q.codebook))


def test_pack_q4x_errors_and_capacity():
    n, k = 2, 256
    codes, s, sel, cb = _random_q4x(n, k, 1)
    d = qx.desc(n, k, 4, 64, qx.QX_Q4X)
    ok = lambda dd=d, **kw: _st(lambda: qx.qx_pack_q4x(dd, **{**dict(codes=codes, scales=s, selectors=sel,
                                                                      codebook=cb), **kw}))
    assert ok() == qx.QX_OK
    assert ok(codes=np.full((n, k), 16, np.uint8)) == qx.QX_E_ARG
    assert ok(selectors=np.full((n, 4), 4, np.uint8)) == qx.QX_E_ARG
    assert ok(dd=qx.desc(n, k, 3, 64, qx.QX_Q4X)) == qx.QX_E_ARG    # the format fixes b = 4
    assert ok(dd=qx.desc(n, k, 4, 128, qx.QX_Q4X)) == qx.QX_E_ARG   # and g = 64
    assert ok(dd=qx.desc(n, k, 4, 64, qx.QX_CODEBOOK)) == qx.QX_E_ARG
    size = oracle.q4x.packed_size(n, k)
    small = np.empty(size - 1, np.uint8)
    assert ok(out=small) == qx.QX_E_SIZE
    # the general packer does not take Q4X descriptors
    assert _st(lambda: qx.qx_pack_layout(d, codes)) == qx.QX_E_ARG
    lib = qx.load()
    sz = ctypes.c_size_t(0)
    P = ctypes.c_void_p
    assert lib.qx_pack_q4x(ctypes.byref(d), None, None, None, None, None, 0, ctypes.byref(sz)) == qx.QX_OK
    assert sz.value == size
    out = np.empty(size, np.uint8)
    assert lib.qx_pack_q4x(ctypes.byref(d), codes.ctypes.data_as(P), None, sel.ctypes.data_as(P),
                           cb.ctypes.data_as(P), out.ctypes.data_as(P), size, ctypes.byref(sz)) == qx.QX_E_ARG


def test_q4x_device_calls_reject_before_launch():
    lib = qx.load()
    d = qx.desc(4, 128, 4, 64, qx.QX_Q4X)
    P = ctypes.c_void_p
    assert lib.qx_gemm(ctypes.byref(d), P(16), 4, None, P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemm(ctypes.byref(d), P(16), -1, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemv(ctypes.byref(d), None, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_dequant(ctypes.byref(d), P(8), 0, P(16), None) == qx.QX_E_ARG
    bad = qx.desc(4, 128, 4, 32, qx.QX_Q4X)
    assert lib.qx_gemv(ctypes.byref(bad), P(16), P(16), P(16), None) == qx.QX_E_ARG


def test_gemv_a8_rejects_before_launch():
    lib = qx.load()
    P = ctypes.c_void_p
    for kind, bits, group in ((qx.QX_CODEBOOK, 3, 128), (qx.QX_Q4X, 4, 64)):
        d = qx.desc(4, 128, bits, group, kind)  # supported: only argument errors are checked here
        assert lib.qx_gemv_a8(ctypes.byref(d), None, P(16), P(16), None) == qx.QX_E_ARG
        assert lib.qx_gemv_a8(ctypes.byref(d), P(16), P(24), P(16), None) == qx.QX_E_ARG
    for long_k in (qx.desc(4, 89 * 128, 4, 128, qx.QX_UNIFORM), qx.desc(4, 89 * 128, 4, 64, qx.QX_Q4X),
                   qx.desc(4, 89 * 128, 3, 64, qx.QX_CODEBOOK)):
        assert lib.qx_gemv_a8(ctypes.byref(long_k), P(16), P(16), P(16), None) == qx.QX_E_UNSUPPORTED
    d = qx.desc(4, 128, 4, 128, qx.QX_UNIFORM)
    assert lib.qx_gemv_a8(ctypes.byref(d), None, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemv_a8(ctypes.byref(d), P(16), P(24), P(16), None) == qx.QX_E_ARG
    z = qx.desc(0, 128, 4, 128, qx.QX_UNIFORM)
    assert lib.qx_gemv_a8(ctypes.byref(z), None, None, None, None) == qx.QX_OK


def test_a8_gemm_calls_reject_before_launch():
    lib = qx.load()
    P = ctypes.c_void_p
    d = qx.desc(64, 4096, 3, 128, 0)
    assert lib.qx_quantize_a8(4, 4000, P(16), P(16), P(16), None) == qx.QX_E_ARG   # k % 128
    assert lib.qx_quantize_a8(-1, 4096, P(16), P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_quantize_a8(4, 4096, None, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_quantize_a8(4, 4096, P(16), P(24), P(16), None) == qx.QX_E_ARG  # Xq alignment
    assert lib.qx_quantize_a8(4, 4096, P(16), P(16), P(18), None) == qx.QX_E_ARG  # sx alignment
    assert lib.qx_quantize_a8(0, 4096, None, None, None, None) == qx.QX_OK
    for kind, bits, group in ((qx.QX_CODEBOOK, 3, 128), (qx.QX_Q4X, 4, 64)):
        t = qx.desc(64, 4096, bits, group, kind)  # supported: only argument errors are checked here
        assert lib.qx_gemm_a8(ctypes.byref(t), None, 4, P(16), P(16), P(16), None) == qx.QX_E_ARG
        assert lib.qx_gemm_a8(ctypes.byref(t), P(16), 4, P(16), P(18), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemm_a8(ctypes.byref(d), P(16), 4, None, P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemm_a8(ctypes.byref(d), P(16), 4, P(16), P(16), P(17), None) == qx.QX_E_ARG
    assert lib.qx_gemm_a8(ctypes.byref(d), P(16), 65537, P(16), P(16), P(16), None) == qx.QX_E_ARG
    assert lib.qx_gemm_a8(ctypes.byref(d), None, 0, None, None, None, None) == qx.QX_OK


class _FakeTensor:
    """Duck-typed stand-in for a device tensor: the binding's checks run, nothing launches."""

    def __init__(self, dtype, numel, contiguous=True, cuda=True, shape=None):
        self.dtype, self._n, self._c, self.is_cuda = dtype, numel, contiguous, cuda
        self.shape = shape if shape is not None else (numel,)

    def dim(self):
        return len(self.shape)

    def numel(self):
        return self._n

    def element_size(self):
        return 2

    def is_contiguous(self):
        return self._c

    def data_ptr(self):
        raise AssertionError("a pointer was taken: the call would have launched")


def test_binding_checks_tensors_against_the_descriptor():
    torch = pytest.importorskip("torch")
    d = qx.desc(64, 256, 4, 128, 0)
    blob = _FakeTensor(torch.uint8, qx.qx_packed_size(d))
    x = _FakeTensor(torch.float16, 256)
    y = _FakeTensor(torch.float16, 64)
    bad = [
        (_FakeTensor(torch.uint8, qx.qx_packed_size(d) - 1), x, y),    # short blob
        (blob, _FakeTensor(torch.float32, 256), y),                    # x dtype
        (blob, _FakeTensor(torch.float16, 255), y),                    # x too short
        (blob, x, _FakeTensor(torch.float16, 63)),                     # y too short
        (blob, _FakeTensor(torch.float16, 256, contiguous=False), y),  # strided x
        (blob, _FakeTensor(torch.float16, 256, cuda=False), y),        # host x
    ]
    for b, xx, yy in bad:
        with pytest.raises(ValueError):
            qx.qx_gemv(d, b, xx, yy)
    X = _FakeTensor(torch.float16, 4 * 256, shape=(4, 256))
    with pytest.raises(ValueError):
        qx.qx_gemm(d, blob, 4, _FakeTensor(torch.float16, 4 * 255, shape=(4, 255)), _FakeTensor(torch.float16, 256))
    with pytest.raises(ValueError):
        qx.qx_gemm(d, blob, 4, X, _FakeTensor(torch.float16, 4 * 64 - 1))
    with pytest.raises(ValueError):
        qx.qx_gemm_a8(d, blob, 4, _FakeTensor(torch.int8, 4 * 256, shape=(4, 256)), _FakeTensor(torch.float16, 4),
                      _FakeTensor(torch.float16, 4 * 64))


def test_load_imports_torch_before_the_library():
    """libqx and torch must share one HIP runtime: load() imports torch (and with it the
    runtime that owns torch's device memory) before it opens libqx, whatever the caller
    imported first. Run in a fresh interpreter so that nothing has imported torch yet."""
    import subprocess
    import sys
    code = ("import sys\n"
            "import paper_2505_07531_amd as qx\n"
            "assert 'torch' not in sys.modules\n"
            "qx.load()\n"
            "assert 'torch' in sys.modules\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
