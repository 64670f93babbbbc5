"""The host side of libqx under AddressSanitizer + UndefinedBehaviorSanitizer, and
ThreadSanitizer: qx_api.cpp (descriptor checks and the host packers, whose codes
region is split across threads for matrices of 256 rows or more) built with g++
against host-only stand-ins for the kernel launchers, driven over every format
including ragged and multithreaded shapes. The sanitized blobs must equal the
library's byte for byte (and so the oracle's, which test_abi pins). CPU only."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import paper_2505_07531_amd as qx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "paper_2505_07531_amd", "csrc", "qx_api.cpp"),
       os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
       os.path.join(ROOT, "tests", "sanitize", "pack_driver.cpp")]
CASES = [(b, kind, g, n, k, 11 + i) for i, (b, kind, g, n, k) in enumerate(
    [(b, kind, g, n, k) for b in (3, 4) for kind in (0, 1) for g in (32, 64, 128)
     for (n, k) in ((3, 384), (300, 1152))] + [(4, 2, 64, 5, 1152), (4, 2, 64, 260, 2048), (4, 0, 128, 0, 256)])]


def _lcg_stream(seed):
    s = seed
    while True:
        s = (s * 6364136223846793005 + 1442695040888963407) & (2**64 - 1)
        yield s >> 33


def _inputs(b, kind, g, n, k, seed):
    """The driver's draws, in its order."""
    r = _lcg_stream(seed)
    codes = np.array([next(r) % (1 << b) for _ in range(n * k)], np.uint8).reshape(n, k)
    G = k // g
    if kind == 2:
        scales = np.array([0x3000 + next(r) % 0x1000 for _ in range(n * G)], np.uint16).reshape(n, G)
        sel = np.array([next(r) % 4 for _ in range(n * G)], np.uint8).reshape(n, G)
        cb = np.array([next(r) & 0xBBFF for _ in range(64)], np.uint16).reshape(4, 16)
        return qx.qx_pack_q4x(qx.desc(n, k, b, g, kind), codes, scales, sel, cb)
    if kind == 0:
        scales = np.array([0x1800 + next(r) % 0x1000 for _ in range(n * G)], np.uint16).reshape(n, G)
        zs = [0x0000, 0x3C00, 0x4000, 0x4200, 0x4400, 0x4500, 0x4600, 0x4700]
        zeros = np.array([zs[next(r) % 8] for _ in range(n * G)], np.uint16).reshape(n, G)
        return qx.qx_pack_layout(qx.desc(n, k, b, g, kind), codes, scales, zeros)
    cb = np.array([next(r) & 0xBBFF for _ in range(n * G << b)], np.uint16).reshape(n, G, 1 << b)
    return qx.qx_pack_layout(qx.desc(n, k, b, g, kind), codes, codebook=cb)


def _build(tmp, flags, name):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = os.path.join(tmp, name)
    cmd = [gxx, "-O1", "-g", "-std=c++17", *flags, "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__",
           "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"), *SRC, "-o", exe, "-pthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip(f"sanitized build unavailable: {r.stderr[-400:]}")
    return exe


@pytest.mark.parametrize("san", ["address,undefined", "thread"])
def test_sanitized_packer_matches_library(tmp_path, san):
    exe = _build(str(tmp_path), [f"-fsanitize={san}", "-fno-sanitize-recover=all"], "drv")
    out = tmp_path / "blobs"
    out.mkdir()
    args = [exe, str(out)] + [str(v) for c in CASES for v in c]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1",
               TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run(args, capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr[-3000:]
    assert "0 unexpected statuses" in r.stdout
    for i, c in enumerate(CASES):
        got = np.fromfile(out / f"{i}.bin", np.uint8)
        assert np.array_equal(got, _inputs(*c)), c
