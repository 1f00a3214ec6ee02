"""Python access to the plain CPU oracle (``liboracle.so``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the product package.
Arguments are numpy arrays in host memory; every function is argument
marshalling around the C oracle in ``wm_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")
SOURCES = [os.path.join(HERE, "wm_oracle.c")]

CRC32_ZLIB = 0
CRC32C = 1

V_HEADER, V_TABLE, V_RECORD, V_DATA, V_STAGING, V_REVERIFY = 1, 2, 4, 8, 16, 32

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into oracle/liboracle.so."""
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
           "-pthread", *SOURCES, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        u64p = ctypes.POINTER(ctypes.c_uint64)
        L.orc_crc_bitwise.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64]
        L.orc_crc_bitwise.restype = ctypes.c_uint32
        L.orc_crc.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64]
        L.orc_crc.restype = ctypes.c_uint32
        L.orc_checksum_chunks.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64,
                                          ctypes.c_uint32, u32p, u32p,
                                          ctypes.c_int]
        L.orc_checksum_chunks.restype = ctypes.c_int
        L.orc_diff_dirty.argtypes = [u8p, u8p, ctypes.c_uint64, ctypes.c_uint32,
                                     u32p, ctypes.c_int]
        L.orc_diff_dirty.restype = ctypes.c_uint32
        L.orc_payload_bound.argtypes = [ctypes.c_uint64, ctypes.c_uint32,
                                        ctypes.c_uint32]
        L.orc_payload_bound.restype = ctypes.c_uint64
        L.orc_encode.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64,
                                 ctypes.c_uint32, u32p, ctypes.c_uint32, u8p,
                                 ctypes.c_uint64, ctypes.c_int]
        L.orc_encode.restype = ctypes.c_int64
        L.orc_plan_chunk.argtypes = [u8p, ctypes.c_uint32, u32p, u32p, u32p,
                                     u32p, u64p]
        L.orc_plan_chunk.restype = ctypes.c_int
        L.orc_decode_verify.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64,
                                        ctypes.c_uint64, ctypes.c_uint32, u8p,
                                        ctypes.c_uint64, u32p, ctypes.c_uint32,
                                        ctypes.c_int]
        L.orc_decode_verify.restype = ctypes.c_uint32
        L.orc_commit.argtypes = [u8p, ctypes.c_uint64, ctypes.c_uint32, u8p,
                                 u8p, ctypes.c_uint32]
        L.orc_commit.restype = ctypes.c_int
        L.orc_commit_reverify.argtypes = [ctypes.c_int, u8p, ctypes.c_uint64, ctypes.c_uint32,
                                          u8p, u8p, ctypes.c_uint32]
        L.orc_commit_reverify.restype = ctypes.c_uint32
        L.orc_encode_codec.argtypes = [ctypes.c_int, ctypes.c_int, u8p, ctypes.c_uint64,
                                       ctypes.c_uint32, u32p, ctypes.c_uint32, u8p,
                                       ctypes.c_uint64, ctypes.c_int]
        L.orc_encode_codec.restype = ctypes.c_int64
        L.orc_decode_verify_codec.argtypes = [ctypes.c_int, ctypes.c_int, u8p, ctypes.c_uint64,
                                              ctypes.c_uint64, ctypes.c_uint32, u8p,
                                              ctypes.c_uint64, u32p, ctypes.c_uint32,
                                              ctypes.c_int]
        L.orc_decode_verify_codec.restype = ctypes.c_uint32
        L.orc_huffman_lengths.argtypes = [u32p, u8p]
        L.orc_huffman_lengths.restype = ctypes.c_uint32
        L.orc_plan_chunk_v2.argtypes = [u8p, ctypes.c_uint32, u32p, u32p, u32p, u32p, u64p]
        L.orc_plan_chunk_v2.restype = ctypes.c_int
        L.orc_plan_chunk_huf.argtypes = [ctypes.c_int, u8p, ctypes.c_uint32, u32p, u32p, u32p,
                                         u32p, u64p]
        L.orc_plan_chunk_huf.restype = ctypes.c_int
        L.orc_flat_layout.argtypes = [u64p, ctypes.c_uint32, u64p]
        L.orc_flat_layout.restype = ctypes.c_uint64
        L.orc_flatten.argtypes = [ctypes.POINTER(u8p), u64p, ctypes.c_uint32,
                                  u8p]
        L.orc_flatten.restype = None
        L.orc_rehydrate.argtypes = [u8p, ctypes.POINTER(u8p), u64p,
                                    ctypes.c_uint32]
        L.orc_rehydrate.restype = None
        _lib = L
    return _lib


def _bytes(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    return a.reshape(-1).view(np.uint8)


def _p8(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))


def _p32(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))


def crc(kind: int, data) -> int:
    b = _bytes(data)
    return int(lib().orc_crc(kind, _p8(b), b.size))


def crc_bitwise(kind: int, data) -> int:
    b = _bytes(data)
    return int(lib().orc_crc_bitwise(kind, _p8(b), b.size))


def n_chunks(nbytes: int, chunk: int) -> int:
    return (nbytes + chunk - 1) // chunk


def unit(chunk: int) -> int:
    """Bytes per record: the chunk up to 64 KiB, else a 64 KiB tile."""
    return min(chunk, 65536)


def checksum_chunks(kind: int, data, chunk: int = 65536, threads: int = 1):
    """Per-chunk CRCs (uint32 array) and the whole-buffer CRC."""
    b = _bytes(data)
    out = np.zeros(max(n_chunks(b.size, chunk), 1), np.uint32)
    g = np.zeros(1, np.uint32)
    rc = lib().orc_checksum_chunks(kind, _p8(b), b.size, chunk, _p32(out),
                                   _p32(g), threads)
    if rc != 0:
        raise ValueError("orc_checksum_chunks rejected its arguments")
    return out[: n_chunks(b.size, chunk)], int(g[0])


def diff_dirty(cur, prev, chunk: int = 65536, threads: int = 1) -> np.ndarray:
    c, p = _bytes(cur), _bytes(prev)
    assert c.size == p.size
    idx = np.zeros(max(n_chunks(c.size, chunk), 1), np.uint32)
    m = lib().orc_diff_dirty(_p8(c), _p8(p), c.size, chunk, _p32(idx), threads)
    return idx[:m].copy()


def payload_bound(nbytes: int, chunk: int, n_records: int) -> int:
    return int(lib().orc_payload_bound(nbytes, chunk, n_records))


def encode(kind: int, state, chunk: int = 65536, idx=None,
           threads: int = 1, codec: int = 1) -> np.ndarray:
    """Payload bytes (uint8 array of exactly payload_bytes); codec 1 is
    format v1, codec 2 format v2 (Huffman-coded exponents)."""
    b = _bytes(state)
    if idx is None:
        n_rec, pidx = n_chunks(b.size, chunk), None
        idx_arr = None
    else:
        idx_arr = np.ascontiguousarray(idx, dtype=np.uint32)
        n_rec = idx_arr.size
        pidx = _p32(idx_arr) if idx_arr.size else _p32(np.zeros(1, np.uint32))
    cap = payload_bound(b.size, chunk, n_rec)
    out = np.zeros(max(cap, 64), np.uint8)
    n = lib().orc_encode_codec(kind, codec, _p8(b), b.size, chunk, pidx, n_rec,
                               _p8(out), out.size, threads)
    if n < 0:
        raise ValueError(f"orc_encode failed ({n})")
    return out[:n].copy()


def huffman_lengths(counts) -> tuple[np.ndarray, int]:
    """Code lengths of format v2 for 256 symbol counts, and the longest."""
    c = np.ascontiguousarray(counts, dtype=np.uint32)
    assert c.size == 256
    out = np.zeros(256, np.uint8)
    k = lib().orc_huffman_lengths(_p32(c), _p8(out))
    return out, int(k)


def plan_chunk_v2(chunk_bytes, codec: int = 2) -> dict:
    """Plan of one chunk's record in format v2 (codec 2: Huffman-coded
    exponents) or v3 (codec 3: Huffman-coded high bytes)."""
    b = _bytes(chunk_bytes)
    m, k, base, sb = (np.zeros(1, np.uint32) for _ in range(4))
    size = np.zeros(1, np.uint64)
    lib().orc_plan_chunk_huf(codec, _p8(b), b.size, _p32(m), _p32(k), _p32(base), _p32(sb),
                             size.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
    return dict(mode=int(m[0]), k=int(k[0]), base=int(base[0]),
                stream_bytes=int(sb[0]), size=int(size[0]))


def plan_chunk(chunk_bytes) -> dict:
    b = _bytes(chunk_bytes)
    m, k, base, esc = (np.zeros(1, np.uint32) for _ in range(4))
    size = np.zeros(1, np.uint64)
    lib().orc_plan_chunk(_p8(b), b.size, _p32(m), _p32(k), _p32(base),
                         _p32(esc),
                         size.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
    return dict(mode=int(m[0]), k=int(k[0]), base=int(base[0]),
                n_esc=int(esc[0]), size=int(size[0]))


def decode_verify(kind: int, payload, nbytes: int, chunk: int = 65536,
                  staging_cap: int | None = None, threads: int = 1, codec: int = 1):
    """Returns (verdict, staging uint8 array, per-record status array)."""
    p = _bytes(payload)
    if staging_cap is None:
        staging_cap = n_chunks(nbytes, unit(chunk)) * unit(chunk)
    staging = np.zeros(max(staging_cap, 1), np.uint8)
    nst = max(n_chunks(nbytes, unit(chunk)), 1)
    status = np.zeros(nst, np.uint32)
    v = lib().orc_decode_verify_codec(kind, codec, _p8(p), p.size, nbytes, chunk,
                                      _p8(staging), staging_cap, _p32(status), nst,
                                      threads)
    return int(v), staging[:staging_cap], status


def commit(live: np.ndarray, chunk: int, staging, payload, verdict: int) -> int:
    """In-place install into `live` (uint8 array). 0 = installed, 1 = refused."""
    assert live.dtype == np.uint8 and live.flags.c_contiguous
    s, p = _bytes(staging), _bytes(payload)
    return int(lib().orc_commit(_p8(live), live.size, chunk, _p8(s), _p8(p),
                                verdict))


def commit_reverify(kind: int, live: np.ndarray, chunk: int, staging, payload,
                    verdict: int) -> int:
    """Re-verifying install into `live` (uint8 array): returns the verdict
    (the given one if nonzero, else 0 = installed or V_REVERIFY = refused,
    live untouched)."""
    assert live.dtype == np.uint8 and live.flags.c_contiguous
    s, p = _bytes(staging), _bytes(payload)
    return int(lib().orc_commit_reverify(kind, _p8(live), live.size, chunk, _p8(s), _p8(p),
                                         verdict))


def _u64p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))


def flat_layout(sizes) -> tuple[np.ndarray, int]:
    """Offsets of the leaves in the flat buffer and the flat size."""
    b = np.ascontiguousarray(sizes, dtype=np.uint64)
    off = np.zeros(max(b.size, 1), np.uint64)
    total = lib().orc_flat_layout(_u64p(b), b.size, _u64p(off))
    return off[: b.size], int(total)


def _ptr_table(arrays):
    u8p = ctypes.POINTER(ctypes.c_uint8)
    t = (u8p * max(len(arrays), 1))()
    for i, a in enumerate(arrays):
        t[i] = _p8(a)
    return t


def flatten(leaves) -> np.ndarray:
    """Flat bytes of a manifest given as a list of arrays (any dtype)."""
    bs = [_bytes(x) for x in leaves]
    sizes = np.array([b.size for b in bs], np.uint64)
    _, total = flat_layout(sizes)
    flat = np.full(max(total, 1), 0xA5, np.uint8)  # every byte gets written
    lib().orc_flatten(_ptr_table(bs), _u64p(sizes), len(bs), _p8(flat))
    return flat[:total]


def rehydrate(flat, sizes) -> list[np.ndarray]:
    """The leaves (uint8 arrays of the given sizes) held by a flat buffer."""
    f = _bytes(flat)
    sz = np.ascontiguousarray(sizes, dtype=np.uint64)
    _, total = flat_layout(sz)
    if f.size < total:
        raise ValueError("flat buffer smaller than the manifest")
    out = [np.zeros(max(int(s), 1), np.uint8) for s in sz]
    lib().orc_rehydrate(_p8(f), _ptr_table(out), _u64p(sz), sz.size)
    return [o[: int(s)] for o, s in zip(out, sz)]


# ---- pre-copy occupancy model (App. H: the coupon-law derivation) ---------
# w chunk writes, each to one of N chunks drawn uniformly with replacement,
# leave a dirty set whose size is the number of distinct chunks hit.


def occupancy_mean(n: int, w: int) -> float:
    """Expected distinct chunks: N (1 - (1 - 1/N)^w), which the paper writes
    in its large-N form N (1 - e^(-w/N)) (w counted in chunks)."""
    return n * (1.0 - (1.0 - 1.0 / n) ** w)


def occupancy_var(n: int, w: int) -> float:
    """Variance of the distinct count (sum of N dependent indicators)."""
    q1 = (1.0 - 1.0 / n) ** w
    q2 = (1.0 - 2.0 / n) ** w if n > 1 else 0.0
    return n * q1 + n * (n - 1) * q2 - (n * q1) ** 2


def precopy_recursion(n: int, rho: float, n0: int, rounds: int) -> list:
    """Expected dirty chunks per round when the source writes rho chunks per
    chunk shipped: d_0 = n0, d_(k+1) = N (1 - e^(-rho d_k / N))."""
    import math
    d = [float(n0)]
    for _ in range(rounds - 1):
        d.append(n * (1.0 - math.exp(-rho * d[-1] / n)))
    return d
