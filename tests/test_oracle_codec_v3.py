"""Pins of the oracle's format v3 (codec 3): the bf16 byte-plane split of
§6.4's codec paragraph.  Each word's high byte (sign and the exponent's upper
seven bits) is coded with the chunk's own canonical Huffman code (lengths at
most 11) in 512 streams; the low byte (the exponent's lowest bit and the
mantissa) stays raw.  Records are RAW (high-byte plane then low-byte plane)
or HUF.  An independent writer built from the format's definition with zlib
pins the encoder's bytes for both record kinds; payloads round-trip; every
single flipped bit of a small payload aborts; the reading that keeps the low
plane raw is checked against its measured entropy."""
import struct
import zlib

import numpy as np
import pytest

import oracle

CH = 65536
MAXLEN = 11


def bf16_state(rng, n_words, sigma=0.5):
    x = rng.standard_normal(n_words) * np.exp(sigma * rng.standard_normal(n_words // 64 + 1)).repeat(64)[:n_words]
    return (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)


def _pad16(x):
    return -(-x // 16) * 16


def _canonical(lens):
    codes, code, bl = {}, 0, [0] * 16
    for ln in lens:
        bl[ln] += 1
    bl[0] = 0
    nxt = [0] * 16
    for b in range(1, 16):
        code = (code + bl[b - 1]) << 1
        nxt[b] = code
    for s in range(256):
        if lens[s]:
            codes[s] = nxt[lens[s]]
            nxt[lens[s]] += 1
    return codes


def _record(state: np.ndarray, huf: bool) -> bytes:
    """One v3 record of the words in state, HUF (whatever its size) or RAW,
    from the format's definition (CRC-32 of zlib for the header's CRC)."""
    w = state.view(np.uint16)
    n = w.size
    hi = (w >> 8).astype(np.int64)
    lo = (w & 0xFF).astype(np.uint8)
    if not huf:
        hdr = struct.pack("<BBBBII", 0, 0, 0, 0, n, 0)
        body = hi.astype(np.uint8).tobytes() + bytes(_pad16(n) - n)
        body += lo.tobytes() + bytes(_pad16(n) - n)
        return hdr + struct.pack("<I", zlib.crc32(hdr)) + body
    lens, k = oracle.huffman_lengths(np.bincount(hi, minlength=256))
    codes = _canonical([int(x) for x in lens])
    streams, sbytes = b"", []
    for s in range(512):
        bits = []
        for i in range(64):
            wi = (8 * (s // 64) + i // 8) * 512 + 8 * (s % 64) + i % 8
            if wi < n:
                ln, c = int(lens[hi[wi]]), codes[int(hi[wi])]
                bits += [(c >> b) & 1 for b in range(ln - 1, -1, -1)]
        out = bytearray(-(-len(bits) // 8))
        for j, bit in enumerate(bits):
            out[j // 8] |= bit << (j % 8)
        sbytes.append(len(out))
        streams += bytes(out)
    nib = bytearray(128)
    for s in range(256):
        nib[s // 2] |= int(lens[s]) << (4 * (s % 2))
    hdr = struct.pack("<BBBBII", 2, k, 0, 0, n, len(streams))
    rec = hdr + struct.pack("<I", zlib.crc32(hdr)) + bytes(nib) + bytes(sbytes)
    rec += streams + bytes(_pad16(len(streams)) - len(streams))
    rec += lo.tobytes() + bytes(_pad16(n) - n)
    return rec


def _payload(state: np.ndarray, huf: bool) -> bytes:
    """One-chunk v3 payload (CRC-32 kind) around _record."""
    rec = _record(state, huf)
    table = struct.pack("<IIQ", 0, zlib.crc32(state.tobytes()), 64)
    total = 64 + len(rec) + 16
    h = b"WMV3" + struct.pack("<HBBIIQIIQII", 3, 0, 3, CH, 1, state.size, 1, 1, total,
                              zlib.crc32(state.tobytes()), zlib.crc32(table)) + bytes(12)
    h += struct.pack("<I", zlib.crc32(h))
    return h + rec + table


def test_independent_writer_matches_the_oracle_huf():
    rng = np.random.default_rng(21)
    st = bf16_state(rng, 3000)
    want = oracle.encode(0, st, CH, None, 1, codec=3)
    assert want[64] == 2  # HUF chosen
    assert _payload(st, True) == want.tobytes()


def test_independent_writer_matches_the_oracle_raw():
    rng = np.random.default_rng(22)
    st = rng.integers(0, 1 << 16, 3000, dtype=np.uint16).view(np.uint8)
    want = oracle.encode(0, st, CH, None, 1, codec=3)
    assert want[64] == 0  # RAW chosen for uniform random words
    assert _payload(st, False) == want.tobytes()


def test_planes_differ_from_format_v2():
    """v3 codes the high byte, v2 the exponent: the same words give
    different code lengths, and a constant chunk's base is its high byte."""
    n = CH // 2
    const = np.full(n, 0x3F80, np.uint16).view(np.uint8)  # 1.0 everywhere
    assert oracle.plan_chunk_v2(const, codec=3) == dict(mode=2, k=0, base=0x3F,
                                                        stream_bytes=0, size=16 + n)
    assert oracle.plan_chunk_v2(const, codec=2)["base"] == 127
    # +-1.0 alternating: one exponent (v2 k = 0) but two high bytes (v3 k = 1)
    alt = np.tile(np.array([0x3F80, 0xBF80], np.uint16), n // 2).view(np.uint8)
    p2, p3 = oracle.plan_chunk_v2(alt, codec=2), oracle.plan_chunk_v2(alt, codec=3)
    assert p2["k"] == 0 and p3["k"] == 1
    assert p3["stream_bytes"] == n // 8  # one bit per word, 64 words per stream


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("n_chunks_", [1, 3])
def test_round_trip_and_cross_rejection(kind, n_chunks_):
    rng = np.random.default_rng(23 + kind)
    st = bf16_state(rng, n_chunks_ * CH // 2 - 2768)  # short last chunk
    p3 = oracle.encode(kind, st, CH, None, 4, codec=3)
    v, stg, rs = oracle.decode_verify(kind, p3, st.size, CH, None, 4, codec=3)
    assert v == 0 and not rs.any()
    assert np.array_equal(stg[: st.size], st)
    assert p3[:4].tobytes() == b"WMV3" and p3[7] == 3
    p2 = oracle.encode(kind, st, CH, None, 4, codec=2)
    for other, codec in ((p2, 3), (p3, 2), (p3, 1)):
        assert oracle.decode_verify(kind, other, st.size, CH, None, 4, codec=codec)[0] == 1


def test_dirty_list_and_large_chunks():
    rng = np.random.default_rng(24)
    st = bf16_state(rng, 5 * CH // 2)
    idx = np.array([1, 3, 4], np.uint32)
    p = oracle.encode(0, st, CH, idx, 2, codec=3)
    v, stg, _ = oracle.decode_verify(0, p, st.size, CH, None, 2, codec=3)
    assert v == 0
    for r, c in enumerate(idx):
        assert np.array_equal(stg[r * CH:(r + 1) * CH], st[c * CH:(c + 1) * CH])
    # chunks above 64 KiB ship as tiles, like the other formats
    p2 = oracle.encode(0, st, 2 * CH, None, 2, codec=3)
    v, stg, _ = oracle.decode_verify(0, p2, st.size, 2 * CH, None, 2, codec=3)
    assert v == 0 and np.array_equal(stg[: st.size], st)


def test_stream_bytes_within_entropy_bounds():
    rng = np.random.default_rng(25)
    # normal values with magnitudes clipped to [2^-6, 2^6): a dozen
    # exponents of either sign, no code longer than 11 bits
    x = rng.standard_normal(CH // 2).astype(np.float32) * 3
    x = np.sign(x) * np.clip(np.abs(x), 2.0 ** -6, 63.0)
    st = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    w = st.view(np.uint16)
    counts = np.bincount(w >> 8, minlength=256)
    lens, k = oracle.huffman_lengths(counts)
    assert k < MAXLEN
    p = counts[counts > 0] / w.size
    H = -(p * np.log2(p)).sum()
    bits = int((counts * lens).sum())
    assert H * w.size <= bits <= (H + 1) * w.size
    plan = oracle.plan_chunk_v2(st, codec=3)
    assert plan["mode"] == 2 and plan["k"] == k
    assert bits / 8 <= plan["stream_bytes"] <= bits / 8 + 512
    assert plan["size"] == 16 + 128 + 512 + _pad16(plan["stream_bytes"]) + w.size


def test_low_plane_is_near_eight_bits():
    """The reading behind keeping the low plane raw: on a KV-cache-like
    chunk its empirical entropy is within 1% of 8 bits, so a code for it
    could remove at most about 1% of the plane."""
    rng = np.random.default_rng(26)
    st = bf16_state(rng, 4 * CH // 2)
    lo = st.view(np.uint16) & 0xFF
    p = np.bincount(lo, minlength=256) / lo.size
    p = p[p > 0]
    assert -(p * np.log2(p)).sum() > 7.92


def test_every_single_bit_flip_aborts():
    rng = np.random.default_rng(27)
    st = bf16_state(rng, 1500, sigma=2.0)  # one short chunk of 3000 bytes
    p = oracle.encode(0, st, CH, None, 1, codec=3)
    assert p[64] == 2  # the record is HUF
    bad = p.copy()
    missed = []
    for i in range(p.size * 8):
        bad[i // 8] ^= 1 << (i % 8)
        if oracle.decode_verify(0, bad, st.size, CH, None, 1, codec=3)[0] == 0:
            missed.append(i)
        bad[i // 8] ^= 1 << (i % 8)
    assert not missed


def test_a_huf_record_longer_than_raw_is_rejected():
    rng = np.random.default_rng(28)
    st = rng.integers(0, 1 << 16, 3000, dtype=np.uint16).view(np.uint8)
    p = np.frombuffer(_payload(st, True), np.uint8)
    v, _, status = oracle.decode_verify(0, p, st.size, CH, None, 1, codec=3)
    assert v == 4 and status[0] == 4
