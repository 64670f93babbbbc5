"""Python binding of libqx (include/qx.h): group-wise 3/4-bit quantized weights,
dequantized and multiplied by fp16 activations on an MI355X.

Argument marshalling only: every step of the path runs in the library's HIP
kernels. PyTorch supplies device memory and streams. If the library is not
built, ``load()`` builds it in-tree with hipcc; if it cannot be loaded, every
call raises -- there is no fallback.

Functions keep the C names:
  qx_pack_layout(desc, codes, scales=None, zeros=None, codebook=None) -> uint8 numpy blob
  qx_pack_q4x(desc, codes, scales, selectors, codebook) -> uint8 numpy blob
  qx_dequant(desc, packed, out_kind, out, stream=None)
  qx_gemv(desc, packed, x, y, stream=None)
  qx_gemv_a8(desc, packed, x, y, stream=None)
  qx_gemm(desc, packed, m, X, Y, stream=None)
  qx_quantize_a8(m, k, X, Xq, sx, stream=None)
  qx_gemm_a8(desc, packed, m, Xq, sx, Y, stream=None)
  qx_status_str(status)
Tensor arguments are torch CUDA tensors (HIP device memory); ``stream`` is a
torch stream (default: the current stream). Before a device call the binding
checks each tensor against the descriptor (device, dtype, contiguity, element
count) and raises ValueError without launching anything when one does not fit.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from . import _build

QX_UNIFORM, QX_CODEBOOK, QX_Q4X = 0, 1, 2
QX_OUT_F16, QX_OUT_CODES = 0, 1
QX_OK, QX_E_ARG, QX_E_UNSUPPORTED, QX_E_SIZE, QX_E_HIP = 0, -1, -2, -3, -4

LIB_PATH = _build.LIB


class QxDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("group", ctypes.c_int32), ("kind", ctypes.c_int32), ("flags", ctypes.c_uint32)]

    def __repr__(self):
        return (f"QxDesc(n={self.n}, k={self.k}, bits={self.bits}, group={self.group}, "
                f"kind={self.kind}, flags={self.flags})")


def desc(n: int, k: int, bits: int, group: int, kind: int, flags: int = 0) -> QxDesc:
    return QxDesc(n, k, bits, group, kind, flags)


class QxError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {qx_status_str(status)} ({status})")


_lib = None


def build() -> str:
    """Compile libqx.so for gfx950 in-tree (always recompiles)."""
    global _lib
    _lib = None
    return _build.build()


def load():
    """The loaded libqx (ctypes.CDLL); builds it first if it is not there."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            _build.build()
        try:  # torch's HIP runtime first, so that libqx binds to the one that owns torch's memory
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        P, sz = ctypes.c_void_p, ctypes.c_size_t
        D = ctypes.POINTER(QxDesc)
        L.qx_pack_layout.argtypes = [D, P, P, P, P, P, sz, ctypes.POINTER(sz)]
        L.qx_pack_layout.restype = ctypes.c_int
        L.qx_pack_q4x.argtypes = [D, P, P, P, P, P, sz, ctypes.POINTER(sz)]
        L.qx_pack_q4x.restype = ctypes.c_int
        L.qx_dequant.argtypes = [D, P, ctypes.c_int, P, P]
        L.qx_dequant.restype = ctypes.c_int
        L.qx_gemv.argtypes = [D, P, P, P, P]
        L.qx_gemv.restype = ctypes.c_int
        L.qx_gemv_a8.argtypes = [D, P, P, P, P]
        L.qx_gemv_a8.restype = ctypes.c_int
        L.qx_gemm.argtypes = [D, P, ctypes.c_int32, P, P, P]
        L.qx_gemm.restype = ctypes.c_int
        L.qx_quantize_a8.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P]
        L.qx_quantize_a8.restype = ctypes.c_int
        L.qx_gemm_a8.argtypes = [D, P, ctypes.c_int32, P, P, P, P]
        L.qx_gemm_a8.restype = ctypes.c_int
        L.qx_status_str.argtypes = [ctypes.c_int]
        L.qx_status_str.restype = ctypes.c_char_p
        _lib = L
    return _lib


def qx_status_str(status: int) -> str:
    return load().qx_status_str(int(status)).decode()


def _np_ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(st: int, where: str):
    if st != QX_OK:
        raise QxError(st, where)


def qx_packed_size(d: QxDesc) -> int:
    size = ctypes.c_size_t(0)
    _check(load().qx_pack_layout(ctypes.byref(d), None, None, None, None, None, 0,
                                 ctypes.byref(size)), "qx_pack_layout")
    return size.value


def qx_pack_layout(d: QxDesc, codes: np.ndarray, scales=None, zeros=None, codebook=None,
                   out: Optional[np.ndarray] = None) -> np.ndarray:
    """Packed blob (host uint8 array) of codes [n][k] and binary16 tables."""
    def c(a, dt):
        return None if a is None else np.ascontiguousarray(a, dtype=dt)
    codes, scales, zeros, codebook = c(codes, np.uint8), c(scales, np.uint16), c(zeros, np.uint16), \
        c(codebook, np.uint16)
    total = qx_packed_size(d)
    if out is None:
        out = np.empty(total, np.uint8)
    size = ctypes.c_size_t(0)
    _check(load().qx_pack_layout(ctypes.byref(d), _np_ptr(codes), _np_ptr(scales), _np_ptr(zeros),
                                 _np_ptr(codebook), _np_ptr(out), out.nbytes, ctypes.byref(size)),
           "qx_pack_layout")
    return out[:size.value]


def qx_pack_q4x(d: QxDesc, codes: np.ndarray, scales, selectors, codebook,
                out: Optional[np.ndarray] = None) -> np.ndarray:
    """Q4X blob (host uint8 array): codes [n][k], scales [n][k/64] (binary16 bits),
    selectors [n][k/64] (< 4), codebook [4][16] (binary16 bits)."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint16)
    selectors = np.ascontiguousarray(selectors, dtype=np.uint8)
    codebook = np.ascontiguousarray(codebook, dtype=np.uint16)
    size = ctypes.c_size_t(0)
    L = load()
    _check(L.qx_pack_q4x(ctypes.byref(d), None, None, None, None, None, 0, ctypes.byref(size)),
           "qx_pack_q4x")
    if out is None:
        out = np.empty(size.value, np.uint8)
    _check(L.qx_pack_q4x(ctypes.byref(d), _np_ptr(codes), _np_ptr(scales), _np_ptr(selectors),
                         _np_ptr(codebook), _np_ptr(out), out.nbytes, ctypes.byref(size)), "qx_pack_q4x")
    return out[:size.value]


def _chk(t, name: str, dtype, numel: int):
    """Check that `t` is a contiguous device tensor of `dtype` (None: any) holding at least
    `numel` elements (the kernels read and write exactly the sizes the descriptor implies)."""
    if t is None:
        raise ValueError(f"{name}: a device tensor is required")
    if not t.is_cuda:
        raise ValueError(f"{name}: device tensors required")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {numel} needed")


def _ptrs(*tensors):
    """Device pointers, taken only once every argument has been checked."""
    return [None if t is None else ctypes.c_void_p(t.data_ptr()) for t in tensors]


def qx_blob_size(d: QxDesc) -> int:
    """Bytes of the packed blob of `d` (any kind)."""
    size = ctypes.c_size_t(0)
    L = load()
    fn = L.qx_pack_q4x if d.kind == QX_Q4X else L.qx_pack_layout
    _check(fn(ctypes.byref(d), None, None, None, None, None, 0, ctypes.byref(size)), "packed size")
    return size.value


def _chk_packed(d: QxDesc, packed):
    import torch
    _chk(packed, "packed", torch.uint8, qx_blob_size(d))


def _rows(X, m: int, k: int, name: str):
    if X is not None and X.dim() == 2 and (X.shape[0] < m or X.shape[1] != k):
        raise ValueError(f"{name}: shape {tuple(X.shape)}, expected ({m}, {k})")


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def qx_dequant(d: QxDesc, packed, out_kind: int, out, stream=None) -> None:
    import torch
    _chk_packed(d, packed)
    _chk(out, "out", torch.float16 if out_kind == QX_OUT_F16 else torch.uint8, d.n * d.k)
    _check(load().qx_dequant(ctypes.byref(d), *_ptrs(packed), out_kind, *_ptrs(out), _stream(stream)),
           "qx_dequant")


def qx_gemv(d: QxDesc, packed, x, y, stream=None) -> None:
    import torch
    _chk_packed(d, packed)
    _chk(x, "x", torch.float16, d.k)
    _chk(y, "y", torch.float16, d.n)
    _check(load().qx_gemv(ctypes.byref(d), *_ptrs(packed, x, y), _stream(stream)), "qx_gemv")


def qx_gemv_a8(d: QxDesc, packed, x, y, stream=None) -> None:
    import torch
    _chk_packed(d, packed)
    _chk(x, "x", torch.float16, d.k)
    _chk(y, "y", torch.float16, d.n)
    _check(load().qx_gemv_a8(ctypes.byref(d), *_ptrs(packed, x, y), _stream(stream)), "qx_gemv_a8")


def qx_gemm(d: QxDesc, packed, m: int, X, Y, stream=None) -> None:
    import torch
    m = int(m)
    _chk_packed(d, packed)
    _rows(X, m, d.k, "X")
    _chk(X, "X", torch.float16, m * d.k)
    _chk(Y, "Y", torch.float16, m * d.n)
    p, x, y = _ptrs(packed, X, Y)
    _check(load().qx_gemm(ctypes.byref(d), p, m, x, y, _stream(stream)), "qx_gemm")


def qx_quantize_a8(m: int, k: int, X, Xq, sx, stream=None) -> None:
    import torch
    m, k = int(m), int(k)
    _chk(X, "X", torch.float16, m * k)
    _chk(Xq, "Xq", torch.int8, m * k)
    _chk(sx, "sx", torch.float32, m)
    _check(load().qx_quantize_a8(m, k, *_ptrs(X, Xq, sx), _stream(stream)), "qx_quantize_a8")


def qx_gemm_a8(d: QxDesc, packed, m: int, Xq, sx, Y, stream=None) -> None:
    import torch
    m = int(m)
    _chk_packed(d, packed)
    _rows(Xq, m, d.k, "Xq")
    _chk(Xq, "Xq", torch.int8, m * d.k)
    _chk(sx, "sx", torch.float32, m)
    _chk(Y, "Y", torch.float16, m * d.n)
    p, xq, s_, y = _ptrs(packed, Xq, sx, Y)
    _check(load().qx_gemm_a8(ctypes.byref(d), p, m, xq, s_, y, _stream(stream)), "qx_gemm_a8")


def quantize_a8(X, stream=None):
    """(Xq int8 [m][k], sx fp32 [m]) of an fp16 [m][k] device tensor."""
    import torch
    m, k = X.shape
    Xq = torch.empty((m, k), dtype=torch.int8, device=X.device)
    sx = torch.empty(m, dtype=torch.float32, device=X.device)
    qx_quantize_a8(m, k, X, Xq, sx, stream)
    return Xq, sx


# ------------------------------------------------------------- conveniences
class PackedWeight:
    """A packed matrix resident in device memory, with its descriptor."""

    def __init__(self, d: QxDesc, blob: np.ndarray, device="cuda"):
        import torch
        self.desc = d
        self.nbytes = int(blob.size)
        self.data = torch.from_numpy(np.ascontiguousarray(blob)).to(device)

    @classmethod
    def from_quant(cls, q, device="cuda") -> "PackedWeight":
        """From an object with n, k, bits, group, kind, codes, scales, zeros, codebook
        (and selectors for Q4X)."""
        d = desc(q.n, q.k, q.bits, q.group, q.kind)
        if q.kind == QX_Q4X:
            return cls(d, qx_pack_q4x(d, q.codes, q.scales, q.selectors, q.codebook), device)
        return cls(d, qx_pack_layout(d, q.codes, q.scales, q.zeros, q.codebook), device)

    def dequant(self, out_kind: int = QX_OUT_F16, stream=None):
        import torch
        dt = torch.float16 if out_kind == QX_OUT_F16 else torch.uint8
        out = torch.empty((self.desc.n, self.desc.k), dtype=dt, device=self.data.device)
        qx_dequant(self.desc, self.data, out_kind, out, stream)
        return out

    def gemv(self, x, y=None, stream=None):
        import torch
        if y is None:
            y = torch.empty(self.desc.n, dtype=torch.float16, device=x.device)
        qx_gemv(self.desc, self.data, x, y, stream)
        return y

    def gemm_a8(self, Xq, sx, Y=None, stream=None):
        import torch
        m = Xq.shape[0]
        if Y is None:
            Y = torch.empty((m, self.desc.n), dtype=torch.float16, device=Xq.device)
        qx_gemm_a8(self.desc, self.data, m, Xq, sx, Y, stream)
        return Y

    def gemv_a8(self, x, y=None, stream=None):
        import torch
        if y is None:
            y = torch.empty(self.desc.n, dtype=torch.float16, device=x.device)
        qx_gemv_a8(self.desc, self.data, x, y, stream)
        return y

    def gemm(self, X, Y=None, stream=None):
        import torch
        m = X.shape[0]
        if Y is None:
            Y = torch.empty((m, self.desc.n), dtype=torch.float16, device=X.device)
        qx_gemm(self.desc, self.data, m, X, Y, stream)
        return Y
