"""Pins for the oracle's CRC (no GPU).

The oracle's CRC is checked against things other than itself: published check
values and RFC 3720 vectors (tests/golden/crc_vectors.txt), Python's zlib for
the zlib polynomial, and the x86 SSE4.2 crc32 instruction (a hardware
implementation of CRC-32C) through a helper compiled here.  Together these
catch a wrong polynomial, a wrong reflection, a wrong init/xorout or a wrong
byte order.  The checksum is the per-chunk CRC of §4 "Sufficiency" and §6.5
(zlib's CRC; CRC-32C selectable).
"""
import ctypes
import os
import subprocess
import zlib

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "crc_vectors.txt")


def golden_vectors():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            kind, msg, want = line.split()
            data = b"" if msg == "-" else bytes.fromhex(msg)
            rows.append((int(kind), data, int(want, 16)))
    return rows


@pytest.mark.parametrize("kind,data,want", golden_vectors())
def test_published_vectors(kind, data, want):
    arr = np.frombuffer(data, np.uint8) if data else np.zeros(0, np.uint8)
    assert oracle.crc_bitwise(kind, arr) == want
    assert oracle.crc(kind, arr) == want


def test_zlib_crc32_random_buffers():
    rng = np.random.default_rng(1234)
    for n in [1, 2, 3, 7, 16, 63, 64, 65, 1000, 4096, 65536, 65537, 300001]:
        buf = rng.integers(0, 256, n, dtype=np.uint8)
        assert oracle.crc(0, buf) == zlib.crc32(buf.tobytes())
    # the bitwise definition agrees with the table form
    buf = rng.integers(0, 256, 5000, dtype=np.uint8)
    for kind in (0, 1):
        assert oracle.crc_bitwise(kind, buf) == oracle.crc(kind, buf)


SSE_SRC = r"""
#include <nmmintrin.h>
#include <stdint.h>
uint32_t hw_crc32c(const uint8_t* p, uint64_t n) {
  uint32_t c = 0xFFFFFFFFu;
  for (uint64_t i = 0; i < n; i++) c = _mm_crc32_u8(c, p[i]);
  return c ^ 0xFFFFFFFFu;
}
"""


def _has_sse42():
    try:
        with open("/proc/cpuinfo") as f:
            return "sse4_2" in f.read()
    except OSError:
        return False


@pytest.mark.skipif(not _has_sse42(), reason="host lacks SSE4.2")
def test_crc32c_against_sse42_instruction(tmp_path):
    src = tmp_path / "hw.c"
    src.write_text(SSE_SRC)
    so = tmp_path / "hw.so"
    subprocess.run(["gcc", "-O2", "-msse4.2", "-shared", "-fPIC", str(src),
                    "-o", str(so)], check=True)
    hw = ctypes.CDLL(str(so))
    hw.hw_crc32c.restype = ctypes.c_uint32
    hw.hw_crc32c.argtypes = [ctypes.c_void_p, ctypes.c_uint64]
    rng = np.random.default_rng(99)
    for n in [0, 1, 5, 31, 32, 33, 4096, 65536, 100003]:
        buf = rng.integers(0, 256, n, dtype=np.uint8)
        want = hw.hw_crc32c(buf.ctypes.data, n)
        assert oracle.crc(1, buf) == want


def test_affine_property():
    """crc(a^b^c) = crc(a)^crc(b)^crc(c) for equal lengths (init and xorout
    cancel in an odd number of terms): a structural invariant of any CRC."""
    rng = np.random.default_rng(5)
    for kind in (0, 1):
        a, b, c = (rng.integers(0, 256, 777, dtype=np.uint8) for _ in range(3))
        assert oracle.crc(kind, a ^ b ^ c) == (
            oracle.crc(kind, a) ^ oracle.crc(kind, b) ^ oracle.crc(kind, c))


def test_checksum_chunks_and_global():
    rng = np.random.default_rng(7)
    chunk = 4096
    for n in [0, 1, 4095, 4096, 4097, 3 * 4096, 3 * 4096 + 123]:
        buf = rng.integers(0, 256, n, dtype=np.uint8)
        for threads in (1, 3):
            crcs, g = oracle.checksum_chunks(0, buf, chunk, threads)
            assert g == zlib.crc32(buf.tobytes())
            want = [zlib.crc32(buf[i:i + chunk].tobytes())
                    for i in range(0, n, chunk)]
            assert crcs.tolist() == want
