"""Pins of the oracle's format v2 (codec 2): per-chunk canonical Huffman
codes of the bf16 exponent plane (the plane that carries the redundancy,
§6.4), code lengths at most 11, 512 streams per chunk.  The Huffman lengths
are checked against an independent optimal-cost computation, the Kraft
equality and a hand-worked example; payloads round-trip and every single
flipped bit of a small payload aborts."""
import heapq
import math

import numpy as np
import pytest

import oracle

CH = 65536
MAXLEN = 11


def optimal_cost(counts):
    """Total bits of an optimal prefix code (sum of all merge weights)."""
    h = [c for c in counts if c > 0]
    if len(h) <= 1:
        return 0
    heapq.heapify(h)
    cost = 0
    while len(h) > 1:
        a, b = heapq.heappop(h), heapq.heappop(h)
        cost += a + b
        heapq.heappush(h, a + b)
    return cost


def test_hand_worked_lengths():
    # counts a=5 (sym 10), b=2 (sym 20), c=1 (sym 30), d=1 (sym 40): merge
    # c+d (2); b and that node tie at 2 and the leaf goes first, merge to 4;
    # then 4 and a=5: lengths a 1, b 2, c 3, d 3
    counts = np.zeros(256, np.uint32)
    counts[[10, 20, 30, 40]] = [5, 2, 1, 1]
    lens, k = oracle.huffman_lengths(counts)
    assert k == 3
    assert {i: int(lens[i]) for i in np.nonzero(lens)[0]} == {10: 1, 20: 2, 30: 3, 40: 3}


@pytest.mark.parametrize("seed", range(40))
def test_lengths_are_optimal_and_complete(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(2, 40))
    counts = np.zeros(256, np.uint32)
    syms = rng.choice(256, m, replace=False)
    counts[syms] = rng.integers(1, 5000, m)
    lens, k = oracle.huffman_lengths(counts)
    assert set(np.nonzero(lens)[0]) == set(syms)
    assert sum(2.0 ** -int(lens[s]) for s in syms) == 1.0  # Kraft equality
    cost = int((counts.astype(np.int64) * lens).sum())
    if k < MAXLEN:  # no length limiting happened: the code is optimal
        assert cost == optimal_cost(counts)
        assert k == int(lens.max())


def test_length_limit():
    # Fibonacci counts force depth ~ number of symbols in an unlimited code
    counts = np.zeros(256, np.uint32)
    fib = [1, 1]
    while len(fib) < 24:
        fib.append(fib[-1] + fib[-2])
    counts[:24] = fib
    lens, k = oracle.huffman_lengths(counts)
    assert k == MAXLEN and int(lens.max()) == MAXLEN
    assert sum(2.0 ** -int(l) for l in lens if l) == 1.0


def min_depth_code(counts):
    """(cost, longest length) of the optimal prefix code with the smallest
    longest length: merges taken from a heap ordered by (weight, subtree
    height, creation order), so among equal weights the shallower subtree
    goes first."""
    h = [(int(c), 0, i) for i, c in enumerate(counts) if c > 0]
    if len(h) <= 1:
        return 0, 0
    heapq.heapify(h)
    seq, cost = len(counts), 0
    while len(h) > 1:
        a, b = heapq.heappop(h), heapq.heappop(h)
        cost += a[0] + b[0]
        heapq.heappush(h, (a[0] + b[0], max(a[1], b[1]) + 1, seq))
        seq += 1
    return cost, h[0][1]


@pytest.mark.parametrize("kind", ["geometric", "pareto", "flat", "log_uniform"])
def test_capped_lengths_match_an_independent_construction(kind):
    # The length limit: counts are halved (rounding up, so no symbol drops
    # out) until the code fits in 11 bits.  Independently: halve until the
    # smallest-longest optimal code fits, then the oracle's lengths must be
    # an optimal code of exactly those counts, with that longest length.  A
    # floor halving, a limit off by one or one halving too many fails here.
    rng = np.random.default_rng({"geometric": 1, "pareto": 2, "flat": 3, "log_uniform": 4}[kind])
    n_capped = 0
    for _ in range(60):
        m = int(rng.integers(2, 120))
        counts = np.zeros(256, np.int64)
        syms = rng.choice(256, m, replace=False)
        if kind == "geometric":
            counts[syms] = rng.geometric(rng.uniform(0.05, 0.5), m)
        elif kind == "pareto":
            counts[syms] = (rng.pareto(rng.uniform(0.3, 1.5), m) * 3 + 1).astype(np.int64)
        elif kind == "flat":
            counts[syms] = rng.integers(1, 4, m)
        else:
            counts[syms] = (2.0 ** rng.uniform(0, 16, m)).astype(np.int64)
        counts = np.minimum(counts, 60000)
        lens, k = oracle.huffman_lengths(counts.astype(np.uint32))
        c, halvings = counts.copy(), 0
        while min_depth_code(c)[1] > MAXLEN:
            c = (c + 1) >> 1
            halvings += 1
        n_capped += halvings > 0
        cost, longest = min_depth_code(c)
        assert set(np.nonzero(lens)[0]) == set(syms)
        assert int((c * lens).sum()) == cost
        assert k == longest == int(lens.max())
        assert sum(2.0 ** -int(x) for x in lens if x) == 1.0
    if kind in ("pareto", "log_uniform"):
        assert n_capped > 10  # the cap is really exercised


def test_degenerate_counts():
    counts = np.zeros(256, np.uint32)
    assert oracle.huffman_lengths(counts)[1] == 0
    counts[77] = 1000
    lens, k = oracle.huffman_lengths(counts)
    assert k == 0 and not lens.any()


def bf16_state(rng, n_words, sigma=1.0):
    x = (rng.standard_normal(n_words) * sigma).astype(np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)


@pytest.mark.parametrize("n_chunks_", [1, 3])
def test_round_trip_and_ratio(n_chunks_):
    rng = np.random.default_rng(1)
    st = bf16_state(rng, n_chunks_ * CH // 2 - 2768)  # short last chunk
    p1 = oracle.encode(0, st, CH, None, 4, codec=1)
    p2 = oracle.encode(0, st, CH, None, 4, codec=2)
    v, stg, rs = oracle.decode_verify(0, p2, st.size, CH, None, 4, codec=2)
    assert v == 0 and not rs.any()
    assert np.array_equal(stg[: st.size], st)
    assert p2[:4].tobytes() == b"WMV2" and p2[7] == 2
    assert p2.size < p1.size
    # a v2 payload is not a v1 payload and vice versa
    assert oracle.decode_verify(0, p2, st.size, CH, None, 4, codec=1)[0] == 1
    assert oracle.decode_verify(0, p1, st.size, CH, None, 4, codec=2)[0] == 1


def test_stream_bits_within_entropy_bounds():
    rng = np.random.default_rng(2)
    # normal values with magnitudes clipped to [2^-6, 2^6): a dozen
    # exponents, no code longer than 11 bits
    x = rng.standard_normal(CH // 2).astype(np.float32) * 3
    x = np.sign(x) * np.clip(np.abs(x), 2.0 ** -6, 63.0)
    st = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    w = st.view(np.uint16)
    e = (w >> 7) & 255
    counts = np.bincount(e, minlength=256)
    lens, k = oracle.huffman_lengths(counts)
    assert k < MAXLEN
    p = counts[counts > 0] / w.size
    H = -(p * np.log2(p)).sum()
    bits = int((counts * lens).sum())
    assert H * w.size <= bits <= (H + 1) * w.size
    plan = oracle.plan_chunk_v2(st)
    # streams are byte-padded each: between the bits and bits + 7 per stream
    assert bits / 8 <= plan["stream_bytes"] <= bits / 8 + 512
    assert plan["mode"] == 2 and plan["k"] == k
    assert plan["size"] == 16 + 128 + 512 + -(-plan["stream_bytes"] // 16) * 16 + w.size


def test_constant_and_random_chunks():
    n = CH // 2
    const = np.full(n, 0x3F80, np.uint16).view(np.uint8)  # 1.0 everywhere
    plan = oracle.plan_chunk_v2(const)
    assert plan == dict(mode=2, k=0, base=127, stream_bytes=0, size=16 + n)
    rng = np.random.default_rng(3)
    rnd = rng.integers(0, 1 << 16, n, dtype=np.uint16).view(np.uint8)
    assert oracle.plan_chunk_v2(rnd) == dict(mode=0, k=0, base=0, stream_bytes=0,
                                             size=16 + 2 * n)
    for st in (const, rnd, np.arange(1 << 16, dtype=np.uint16).view(np.uint8)[:CH]):
        p = oracle.encode(1, st, CH, None, 1, codec=2)
        v, stg, _ = oracle.decode_verify(1, p, st.size, CH, None, 1, codec=2)
        assert v == 0 and np.array_equal(stg[: st.size], st)


def test_dirty_list_payload():
    rng = np.random.default_rng(4)
    st = bf16_state(rng, 5 * CH // 2)
    idx = np.array([1, 3, 4], np.uint32)
    p = oracle.encode(0, st, CH, idx, 2, codec=2)
    v, stg, _ = oracle.decode_verify(0, p, st.size, CH, None, 2, codec=2)
    assert v == 0
    for r, c in enumerate(idx):
        assert np.array_equal(stg[r * CH:(r + 1) * CH], st[c * CH:(c + 1) * CH])


def test_every_single_bit_flip_aborts():
    rng = np.random.default_rng(5)
    st = bf16_state(rng, 1500, sigma=2.0)  # one short chunk of 3000 bytes
    p = oracle.encode(0, st, CH, None, 1, codec=2)
    assert p[64] == 2  # the record is HUF
    bad = p.copy()
    missed = []
    for i in range(p.size * 8):
        bad[i // 8] ^= 1 << (i % 8)
        if oracle.decode_verify(0, bad, st.size, CH, None, 1, codec=2)[0] == 0:
            missed.append(i)
        bad[i // 8] ^= 1 << (i % 8)
    assert not missed


# ---- an independent writer of format v2 HUF records, from the format's
# definition (header, code-length nibbles, stream byte counts, streams,
# sign/mantissa plane), used to pin the oracle's encoder and its rules

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


def _pad16(x):
    return -(-x // 16) * 16


def _huf_payload(state: np.ndarray) -> bytes:
    """One-chunk v2 payload whose record is HUF whatever its size (CRC-32)."""
    import struct
    import zlib
    w = state.view(np.uint16)
    n = w.size
    e = ((w >> 7) & 255).astype(np.int64)
    sm = (((w >> 8) & 0x80) | (w & 0x7F)).astype(np.uint8)
    lens, k = oracle.huffman_lengths(np.bincount(e, minlength=256))
    codes = _canonical([int(x) for x in lens])
    streams, sbytes = b"", []
    for s in range(512):
        bits = []
        for i in range(64):
            wi = (8 * (s // 64) + i // 8) * 512 + 8 * (s % 64) + i % 8
            if wi < n:
                ln, c = int(lens[e[wi]]), codes[int(e[wi])]
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
    rec += sm.tobytes() + bytes(_pad16(n) - n)
    table = struct.pack("<IIQ", 0, zlib.crc32(state.tobytes()), 64)
    total = 64 + len(rec) + 16
    h = b"WMV2" + struct.pack("<HBBIIQIIQII", 2, 0, 2, CH, 1, state.size, 1, 1, total,
                              zlib.crc32(state.tobytes()), zlib.crc32(table)) + bytes(12)
    h += struct.pack("<I", zlib.crc32(h))
    return h + rec + table


def test_independent_writer_matches_the_oracle():
    rng = np.random.default_rng(12)
    x = np.sign(rng.standard_normal(3000)) * np.clip(np.abs(rng.standard_normal(3000) * 3),
                                                      2.0 ** -6, 63.0)
    st = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    want = oracle.encode(0, st, CH, None, 1, codec=2)
    assert want[64] == 2  # HUF chosen
    assert _huf_payload(st) == want.tobytes()


def test_a_huf_record_longer_than_raw_is_rejected():
    # uniform random words: the encoder picks RAW; a HUF record of the same
    # words is well formed in every other respect but longer than RAW
    rng = np.random.default_rng(13)
    st = rng.integers(0, 1 << 16, 3000, dtype=np.uint16).view(np.uint8)
    assert oracle.encode(0, st, CH, None, 1, codec=2)[64] == 0
    p = np.frombuffer(_huf_payload(st), np.uint8)
    v, _, status = oracle.decode_verify(0, p, st.size, CH, None, 1, codec=2)
    assert v == 4 and status[0] == 4
