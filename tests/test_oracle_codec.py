"""Pins for the oracle's payload codec (no GPU).

The codec is this project's payload format v1 (the paper fixes no byte
layout; its codec is lossless, splits bf16 planes and keeps decode inside the
verified envelope: §6.4 codec paragraph).  Pins here do not reuse the oracle's
code paths:
  * round-trip identity on random, constant and all-65536-bit-pattern inputs;
  * closed-form record sizes (constant chunk -> PACK k=0; uniform random
    16-bit words -> RAW);
  * a brute-force argmin over every (k, base) on tiny chunks;
  * escape-index entries counted word by word;
  * hand-built expected bytes for a three-chunk payload (PACK k=0, PACK
    k=2, RAW) and for a two-record payload with escapes (PACK k=5 with
    escapes in four 512-word blocks, PACK k=7 on a short tail), with CRCs
    from zlib.
"""
import struct
import zlib

import numpy as np
import pytest

import oracle

CH = 4096  # smallest legal chunk; keeps brute force cheap


def pad16(x):
    return (x + 15) // 16 * 16


def roundtrip(state_u8, chunk=CH, kind=0, idx=None):
    payload = oracle.encode(kind, state_u8, chunk, idx)
    v, staging, st = oracle.decode_verify(kind, payload, state_u8.size, chunk)
    assert v == 0, (v, st)
    live = np.zeros_like(state_u8) if idx is None else state_u8.copy()
    assert oracle.commit(live, chunk, staging, payload, v) == 0
    return payload, live


@pytest.mark.parametrize("kind", [0, 1])
def test_roundtrip_random_bf16(kind):
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(5 * CH // 2 + 7) *
         np.exp(0.5 * rng.standard_normal(1))).astype(np.float32)
    bf = (x.view(np.uint32) >> 16).astype(np.uint16)
    state = bf.view(np.uint8)
    payload, live = roundtrip(state, kind=kind)
    assert np.array_equal(live, state)
    assert payload.size < state.size  # normal data compresses


def test_roundtrip_all_bit_patterns():
    allw = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    for order in ("sorted", "shuffled"):
        w = allw if order == "sorted" else np.random.default_rng(3).permutation(allw)
        state = w.view(np.uint8)
        _, live = roundtrip(state)
        assert np.array_equal(live, state)


def test_roundtrip_special_values():
    # NaN payloads, +-Inf, +-0, denormals, max finite: bit patterns only
    vals = np.array([0x7FC0, 0x7F81, 0xFFC1, 0x7F80, 0xFF80, 0x0000, 0x8000,
                     0x0001, 0x807F, 0x7F7F, 0xFF7F], np.uint16)
    w = np.resize(vals, CH // 2 * 3)
    state = w.view(np.uint8)
    _, live = roundtrip(state)
    assert np.array_equal(live, state)


def test_constant_chunk_closed_form():
    n = CH // 2
    w = np.full(n, 0x3F80, np.uint16)  # 1.0 everywhere: one exponent, sm = 0
    plan = oracle.plan_chunk(w.view(np.uint8))
    assert plan == dict(mode=1, k=0, base=127, n_esc=0, size=16 + pad16(n))
    payload, live = roundtrip(w.view(np.uint8))
    assert np.array_equal(live, w.view(np.uint8))


def test_random_bits_choose_raw():
    rng = np.random.default_rng(11)
    n = CH // 2
    w = rng.integers(0, 65536, n, dtype=np.uint32).astype(np.uint16)
    plan = oracle.plan_chunk(w.view(np.uint8))
    assert plan["mode"] == 0 and plan["size"] == 16 + 2 * n
    assert plan["k"] == 0 and plan["base"] == 0 and plan["n_esc"] == 0


def brute_force_plan(words):
    """Smallest record over every candidate; ties RAW < k=0 < k=1 < ... < 7,
    and for a given k the smallest base.  Counts escapes word by word."""
    n = len(words)
    e = [(int(w) >> 7) & 255 for w in words]
    best = (16 + 2 * pad16(n), 0, 0, 0, 0)  # size, mode, k, base, n_esc
    if len(set(e)) == 1:
        s = 16 + pad16(n)
        if s < best[0]:
            best = (s, 1, 0, e[0], 0)
    for k in range(1, 8):
        width = (1 << k) - 1
        kbest = None
        for base in range(256):
            esc = sum(1 for x in e if not (base <= x < base + width))
            if kbest is None or esc < kbest[1]:
                kbest = (base, esc)
        base, esc = kbest
        s = 16 + pad16((n * k + 7) // 8) + pad16(2 * ((n + 511) // 512)) + \
            pad16(esc) + pad16(n)
        if s < best[0]:
            best = (s, 1, k, base, esc)
    return dict(size=best[0], mode=best[1], k=best[2], base=best[3],
                n_esc=best[4])


@pytest.mark.parametrize("seed", range(12))
def test_plan_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 400))
    kind = seed % 4
    if kind == 0:  # normal-ish values, a few exponents
        x = rng.standard_normal(n).astype(np.float32) * float(rng.uniform(0.01, 100))
        w = (x.view(np.uint32) >> 16).astype(np.uint16)
    elif kind == 1:  # exponents from a narrow random set
        es = rng.integers(0, 256, int(rng.integers(1, 9)))
        e = rng.choice(es, n)
        w = ((rng.integers(0, 2, n) << 15) | (e << 7) |
             rng.integers(0, 128, n)).astype(np.uint16)
    elif kind == 2:  # random bits
        w = rng.integers(0, 65536, n).astype(np.uint16)
    else:  # near the top and bottom of the exponent range
        e = rng.choice([0, 1, 2, 253, 254, 255], n)
        w = ((e << 7) | rng.integers(0, 128, n)).astype(np.uint16)
    assert oracle.plan_chunk(w.view(np.uint8)) == brute_force_plan(w)


def test_hand_built_payload():
    """Three 4 KiB chunks: chunk 0 constant 1.0 (PACK k=0), chunk 1 exponents
    cycling base..base+2 with k=2, chunk 2 random bits (RAW: exponent plane,
    then sign/mantissa plane).  Expected bytes (header, records, then the
    table) are written out here from the format text, CRCs from zlib."""
    n = CH // 2
    c0 = np.full(n, 0x3F80, np.uint16)
    e1 = 120 + (np.arange(n) % 3)
    sm1 = (np.arange(n) * 37) % 256
    c1 = (((sm1 >> 7) << 15) | (e1 << 7) | (sm1 & 127)).astype(np.uint16)
    c2 = np.random.default_rng(77).integers(0, 65536, n).astype(np.uint16)
    state = np.concatenate([c0, c1, c2]).view(np.uint8)

    def rec(mode, k, base, n_esc, body):
        h = struct.pack("<BBBBII", mode, k, base, 0, n, n_esc)
        return h + struct.pack("<I", zlib.crc32(h)) + body

    r0 = rec(1, 0, 127, 0, bytes(pad16(n)))  # sm plane of zeros
    codes = bytearray(n * 2 // 8)
    for i in range(n):
        code = i % 3
        for b in range(2):
            if (code >> b) & 1:
                j = i * 2 + b
                codes[j // 8] |= 1 << (j % 8)
    index = bytes(16)  # 4 blocks of 512 words, no escapes: four zero u16
    r1 = rec(1, 2, 120, 0, bytes(codes) + index + sm1.astype(np.uint8).tobytes())
    e2 = bytes(int((w >> 7) & 255) for w in c2)
    s2 = bytes(int(((w >> 15) << 7) | (w & 127)) for w in c2)
    r2 = rec(0, 0, 0, 0, e2 + s2)
    table = struct.pack("<IIQ", 0, zlib.crc32(c0.tobytes()), 64)
    table += struct.pack("<IIQ", 1, zlib.crc32(c1.tobytes()), 64 + len(r0))
    table += struct.pack("<IIQ", 2, zlib.crc32(c2.tobytes()), 64 + len(r0) + len(r1))
    total = 64 + len(r0) + len(r1) + len(r2) + len(table)
    head = b"WMV1" + struct.pack("<HBBIIQIIQII", 1, 0, 1, CH, 3, state.size,
                                 3, 1, total, zlib.crc32(state.tobytes()),
                                 zlib.crc32(table)) + bytes(12)
    head += struct.pack("<I", zlib.crc32(head))
    want = head + r0 + r1 + r2 + table
    got = oracle.encode(0, state, CH).tobytes()
    assert len(got) == len(want) == total
    assert got == want


def test_escapes_and_partial_tail():
    # 3 chunks + a short tail; a wide exponent spread forces escapes
    rng = np.random.default_rng(21)
    n = (3 * CH + 1234) // 2
    x = (rng.standard_t(3, n) * 1e3).astype(np.float32)
    w = (x.view(np.uint32) >> 16).astype(np.uint16)
    state = w.view(np.uint8)
    payload, live = roundtrip(state)
    assert np.array_equal(live, state)
    # some record used escapes
    plans = [oracle.plan_chunk(state[i:i + CH]) for i in range(0, state.size, CH)]
    assert any(p["n_esc"] > 0 for p in plans)


def test_dirty_subset_payload_and_install():
    rng = np.random.default_rng(5)
    prev = rng.standard_normal(8 * CH // 2).astype(np.float32)
    prev = (prev.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    cur = prev.copy()
    for c in (1, 4, 7):
        cur[c * CH:(c + 1) * CH] = rng.integers(0, 256, CH, dtype=np.uint8)
    idx = oracle.diff_dirty(cur, prev, CH)
    assert idx.tolist() == [1, 4, 7]
    payload = oracle.encode(0, cur, CH, idx)
    v, staging, _ = oracle.decode_verify(0, payload, cur.size, CH,
                                         staging_cap=3 * CH)
    assert v == 0
    live = prev.copy()
    assert oracle.commit(live, CH, staging, payload, v) == 0
    assert np.array_equal(live, cur)
    # empty dirty set: header-only payload, nothing to install
    payload = oracle.encode(0, cur, CH, np.zeros(0, np.uint32))
    assert payload.size == 64
    v, staging, _ = oracle.decode_verify(0, payload, cur.size, CH)
    assert v == 0


def test_empty_state():
    state = np.zeros(0, np.uint8)
    payload = oracle.encode(0, state, CH)
    assert payload.size == 64
    v, _, _ = oracle.decode_verify(0, payload, 0, CH)
    assert v == 0


def test_thread_count_does_not_change_bytes():
    rng = np.random.default_rng(8)
    x = rng.standard_normal(9 * CH // 2).astype(np.float32)
    state = (x.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    a = oracle.encode(0, state, CH, threads=1)
    b = oracle.encode(0, state, CH, threads=4)
    assert np.array_equal(a, b)


def test_escape_index_counts():
    """Index entry b = escaped words before block b (512 words per block),
    counted here word by word from the record's own codes."""
    rng = np.random.default_rng(12)
    n = 3 * 512 + 100
    e = np.where(rng.random(n) < 0.1, rng.integers(0, 256, n), 127 + rng.integers(0, 3, n))
    w = ((e << 7) | rng.integers(0, 128, n)).astype(np.uint16)
    plan = oracle.plan_chunk(w.view(np.uint8))
    k, base = plan["k"], plan["base"]
    assert plan["mode"] == 1 and k >= 1 and plan["n_esc"] > 0
    payload = oracle.encode(0, np.concatenate([w, np.zeros(CH // 2 - n, np.uint16)]).view(np.uint8)[: 2 * n], CH)
    rec = payload[64:]
    code_bytes = (n * k + 7) // 8
    idx_off = 16 + pad16(code_bytes)
    index = rec[idx_off: idx_off + 2 * 4].view(np.uint16)
    esc = [not (base <= x < base + (1 << k) - 1) for x in e]
    want = [sum(esc[: 512 * b]) for b in range(4)]
    assert index.tolist() == want


def _pack_stream(codes, k):
    """LSB-first k-bit stream: bit b of code i is stream bit i*k + b, stream
    bit j is bit j mod 8 of byte j div 8 (format v1, PACK body)."""
    out = bytearray((len(codes) * k + 7) // 8)
    for i, c in enumerate(codes):
        for b in range(k):
            if (c >> b) & 1:
                j = i * k + b
                out[j // 8] |= 1 << (j % 8)
    return bytes(out)


def _zpad(b):
    return b + bytes(pad16(len(b)) - len(b))


def _pack_record(words, k, base):
    """A PACK record written out field by field from the format text: header,
    codes, escape index (escapes before each 512-word block), escapes in word
    order, sign/mantissa plane; each section zero-padded to 16 bytes."""
    words = [int(w) for w in words]
    n = len(words)
    esc = (1 << k) - 1
    e = [(w >> 7) & 255 for w in words]
    sm = bytes(((w >> 15) << 7) | (w & 127) for w in words)
    codes = [x - base if 0 <= x - base < esc else esc for x in e]
    escaped = [x for x, c in zip(e, codes) if c == esc]
    index = b"".join(struct.pack("<H", sum(1 for c in codes[: 512 * b] if c == esc))
                     for b in range((n + 511) // 512))
    h = struct.pack("<BBBBII", 1, k, base, 0, n, len(escaped))
    h += struct.pack("<I", zlib.crc32(h))
    body = _zpad(_pack_stream(codes, k)) + _zpad(index) + _zpad(bytes(escaped)) + _zpad(sm)
    return h + body, len(escaped)


def test_hand_built_payload_with_escapes():
    """Two records with escapes, expected bytes written here from the format
    text (CRCs from zlib): chunk 0 is PACK k=5 (exponents 100..130, escapes
    three in block 0 and one in each of blocks 1, 2 and 3, so the index
    entries are 0, 3, 4, 5), chunk 1
    a 1,000-byte tail that is PACK k=7 (exponents 60..186 and two escapes).
    The dirty list ships both, so the FULL flag stays clear."""
    n0 = CH // 2
    rng = np.random.default_rng(31)
    e0 = 100 + (np.arange(n0) * 7) % 31
    for pos, val in [(5, 20), (300, 255), (511, 0), (512, 99), (1100, 131), (1900, 7)]:
        e0[pos] = val
    sm0 = rng.integers(0, 256, n0)
    c0 = (((sm0 >> 7) << 15) | (e0 << 7) | (sm0 & 127)).astype(np.uint16)
    n1 = 500
    e1 = 60 + (np.arange(n1) * 5) % 127
    e1[17], e1[499] = 0, 255
    sm1 = rng.integers(0, 256, n1)
    c1 = (((sm1 >> 7) << 15) | (e1 << 7) | (sm1 & 127)).astype(np.uint16)
    state = np.concatenate([c0, c1]).view(np.uint8)
    assert state.size == CH + 1000

    r0, esc0 = _pack_record(c0, 5, 100)
    r1, esc1 = _pack_record(c1, 7, 60)
    assert esc0 == 6 and esc1 == 2
    assert r0[16 + pad16(n0 * 5 // 8): 16 + pad16(n0 * 5 // 8) + 8] == \
        struct.pack("<HHHH", 0, 3, 4, 5)
    assert len(r1) == 16 + pad16((n1 * 7 + 7) // 8) + 16 + 16 + pad16(n1)
    table = struct.pack("<IIQ", 0, zlib.crc32(c0.tobytes()), 64)
    table += struct.pack("<IIQ", 1, zlib.crc32(c1.tobytes()), 64 + len(r0))
    total = 64 + len(r0) + len(r1) + len(table)
    head = b"WMV1" + struct.pack("<HBBIIQIIQII", 1, 0, 1, CH, 2, state.size,
                                 2, 0, total, zlib.crc32(state.tobytes()),
                                 zlib.crc32(table)) + bytes(12)
    head += struct.pack("<I", zlib.crc32(head))
    want = head + r0 + r1 + table
    got = oracle.encode(0, state, CH, np.array([0, 1], np.uint32)).tobytes()
    assert len(got) == len(want) == total
    assert got == want
    v, staging, _ = oracle.decode_verify(0, got, state.size, CH)
    assert v == 0 and np.array_equal(staging[: state.size], state)


def test_reverifying_commit():
    """The re-verifying install checks the state it would produce against
    the source's global CRC: installed (bit-identical to the source) when
    the destination holds the source's previous snapshot, refused with live
    untouched when the destination's base differs in a chunk the payload
    does not carry, or when a staged record changed after verification."""
    rng = np.random.default_rng(9)
    n = 6 * CH + 1000
    prev = rng.integers(0, 256, n, dtype=np.uint8)
    cur = prev.copy()
    for c in (1, 4, 6):  # chunk 6 is the 1,000-byte tail
        lo = c * CH
        cur[lo:min(lo + CH, n)] = rng.integers(0, 256, min(CH, n - lo), dtype=np.uint8)
    idx = oracle.diff_dirty(cur, prev, CH)
    assert idx.tolist() == [1, 4, 6]
    payload = oracle.encode(1, cur, CH, idx)
    v, staging, _ = oracle.decode_verify(1, payload, n, CH, staging_cap=3 * CH)
    assert v == 0
    # the right base: installed, equal to the source
    live = prev.copy()
    assert oracle.commit_reverify(1, live, CH, staging, payload, v) == 0
    assert np.array_equal(live, cur)
    # a base that differs in a clean chunk: the plain commit would report
    # success on a state that is not the source's; the re-verifying one refuses
    live = prev.copy()
    live[2 * CH + 7] ^= 1
    before = live.copy()
    assert oracle.commit_reverify(1, live, CH, staging, payload, v) == oracle.V_REVERIFY
    assert np.array_equal(live, before)
    plain = prev.copy()
    plain[2 * CH + 7] ^= 1
    assert oracle.commit(plain, CH, staging, payload, v) == 0
    assert not np.array_equal(plain, cur)
    # a staged record changed after verification: refused
    bad_staging = staging.copy()
    bad_staging[CH + 5] ^= 0x80
    live = prev.copy()
    assert oracle.commit_reverify(1, live, CH, bad_staging, payload, v) == oracle.V_REVERIFY
    assert np.array_equal(live, prev)
    # a nonzero verdict passes through, nothing installed
    live = prev.copy()
    assert oracle.commit_reverify(1, live, CH, staging, payload, oracle.V_DATA) == oracle.V_DATA
    assert np.array_equal(live, prev)
    # a full ship re-verifies into any live buffer
    full = oracle.encode(0, cur, CH)
    v, st_full, _ = oracle.decode_verify(0, full, n, CH)
    live = np.zeros(n, np.uint8)
    assert oracle.commit_reverify(0, live, CH, st_full, full, v) == 0
    assert np.array_equal(live, cur)
