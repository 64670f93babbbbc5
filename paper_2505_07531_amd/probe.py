"""Binding of libqxprobe.so (include/qx_probe.h): a plain streaming read and an
empty grid, timed by the benchmark as the floor for the libqx kernels.

Tensor arguments are torch CUDA tensors; ``stream`` is a torch stream (default:
the current stream). The library is built in-tree with libqx if it is missing.
"""
from __future__ import annotations

import ctypes
import os

from . import _build

PROBE_LIB_PATH = _build.PROBE_LIB
_lib = None


def load():
    """The loaded libqxprobe (ctypes.CDLL); builds the libraries first if it is not there."""
    global _lib
    if _lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            _build.build()
        L = ctypes.CDLL(PROBE_LIB_PATH)
        P = ctypes.c_void_p
        L.qxp_read.argtypes = [P, ctypes.c_size_t, P, P]
        L.qxp_read.restype = ctypes.c_int
        L.qxp_empty.argtypes = [ctypes.c_int32, P, P]
        L.qxp_empty.restype = ctypes.c_int
        _lib = L
    return _lib


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(st: int, where: str) -> None:
    if st != 0:
        raise RuntimeError(f"{where}: status {st}")


def qxp_read(src, sink, stream=None) -> None:
    """Read every byte of the contiguous device tensor `src` once (its size must be a
    multiple of 16 bytes); `sink` is a device tensor of at least 4 bytes."""
    _check(load().qxp_read(src.data_ptr(), src.numel() * src.element_size(), sink.data_ptr(),
                           _stream(stream)), "qxp_read")


def qxp_empty(blocks: int, sink, stream=None) -> None:
    """Launch `blocks` empty blocks of 256 threads."""
    _check(load().qxp_empty(int(blocks), sink.data_ptr(), _stream(stream)), "qxp_empty")
