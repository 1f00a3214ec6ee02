"""Chunks above 64 KiB: the oracle ships each as its 64 KiB tiles, one record
and one receipt per tile, the chunk staying the unit of dirtiness and of the
per-chunk CRCs.  The pre-copy unit the paper works with is 4 MB (§6.2
Exhibit 2; Appendix H), so the chunk size must reach that far.

Pins, for both formats:
  * the payload for a chunk size C > 64 KiB and a chunk list is the 64 KiB
    payload of the list's tiles except for the header's chunk_bytes,
    n_chunks and header CRC, rebuilt here from the format definition with
    zlib;
  * a table that ships part of a chunk is rejected as a table error, and the
    same records completed to whole chunks are accepted;
  * a 1 MiB chunk holding more escapes than 16 bits count round-trips;
  * the payload bound counts tiles.
"""
import struct
import zlib

import numpy as np
import pytest

import oracle

TILE = 65536
V_TABLE = 2


def bf16_state(nbytes, seed, spread=0.5):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(nbytes // 2) * np.exp(spread * rng.standard_normal(1)))
    w = (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return w.view(np.uint8)


def tiles_of(chunks, chunk, nbytes):
    per = chunk // TILE
    n_tiles = -(-nbytes // TILE)
    return [c * per + j for c in chunks for j in range(per) if c * per + j < n_tiles]


def crc_fn(kind):
    if kind == 0:
        return zlib.crc32
    return lambda b: oracle.crc_bitwise(1, np.frombuffer(bytes(b), np.uint8))


def rebuilt_header(kind, head64, chunk, n_chunks):
    """The 64 KiB payload's header with the chunk size and count of C."""
    h = bytearray(head64)
    struct.pack_into("<II", h, 8, chunk, n_chunks)
    struct.pack_into("<I", h, 60, crc_fn(kind)(bytes(h[:60])) & 0xFFFFFFFF)
    return bytes(h)


@pytest.mark.parametrize("codec", [1, 2, 3])
@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("chunk", [1 << 17, 1 << 18])
def test_payload_is_the_tiles_payload(chunk, kind, codec):
    nbytes = 3 * chunk + 100_000  # a short last chunk of two tiles
    state = bf16_state(nbytes, 11 + kind)
    n = -(-nbytes // chunk)
    for chunks in (None, [1, 3], [0], [3], []):
        big = oracle.encode(kind, state, chunk, chunks, codec=codec)
        tiles = None if chunks is None else tiles_of(chunks, chunk, nbytes)
        small = oracle.encode(kind, state, TILE, tiles, codec=codec)
        assert big.size == small.size
        assert bytes(big[64:]) == bytes(small[64:])
        assert bytes(big[:64]) == rebuilt_header(kind, small[:64], chunk, n)
        # records are units: decode stages tile r at r * 64 KiB
        v, staging, _ = oracle.decode_verify(kind, big, nbytes, chunk, codec=codec)
        assert v == 0
        for r, t in enumerate(range(-(-nbytes // TILE)) if tiles is None else tiles):
            ln = min(TILE, nbytes - t * TILE)
            assert np.array_equal(staging[r * TILE:r * TILE + ln],
                                  state[t * TILE:t * TILE + ln])


@pytest.mark.parametrize("kind", [0, 1])
def test_partial_chunk_tables_are_rejected(kind):
    chunk = 1 << 18  # four tiles
    nbytes = 2 * chunk + 3 * TILE - 4096  # last chunk: three tiles, the last short
    state = bf16_state(nbytes, 5)
    n = 3
    live = np.zeros_like(state)
    cases = {
        (0, 1, 2, 3): 0,            # chunk 0 whole
        (8, 9, 10): 0,              # the short last chunk whole
        (0, 1, 2, 3, 8, 9, 10): 0,
        (0, 1, 2): V_TABLE,         # chunk 0 without its last tile
        (1, 2, 3): V_TABLE,         # chunk 0 without its first tile
        (0, 1, 3): V_TABLE,         # a hole
        (4, 5, 6, 7, 9, 10): V_TABLE,
        (8, 9): V_TABLE,            # the last chunk without its last tile
    }
    for tiles, want in cases.items():
        small = oracle.encode(kind, state, TILE, list(tiles))
        p = small.copy()
        p[:64] = np.frombuffer(rebuilt_header(kind, small[:64], chunk, n), np.uint8)
        v, staging, _ = oracle.decode_verify(kind, p, nbytes, chunk)
        assert v == want, (tiles, v)
        if want == 0:
            got = live.copy()
            assert oracle.commit(got, chunk, staging, p, v) == 0
            for t in tiles:
                sl = slice(t * TILE, min((t + 1) * TILE, nbytes))
                assert np.array_equal(got[sl], state[sl])
            # the other chunks of a zero destination differ from the source
            assert oracle.commit_reverify(kind, live.copy(), chunk, staging, p, v) == 32


def test_escape_counts_beyond_16_bits():
    """Each tile of a 1 MiB chunk holds about 6,500 escapes (one word in five
    far outside the narrow band the rest share): about 105,000 in the chunk,
    more than a 16-bit count holds.  Tiles keep every count in range."""
    chunk = 1 << 20
    rng = np.random.default_rng(8)
    nw = chunk // 2
    e = rng.integers(120, 124, nw)
    far = rng.random(nw) < 0.2
    e[far] = rng.integers(0, 256, far.sum())
    w = ((rng.integers(0, 2, nw) << 15) | (e << 7) | rng.integers(0, 128, nw)).astype(np.uint16)
    state = w.view(np.uint8)
    plans = [oracle.plan_chunk(state[i:i + TILE]) for i in range(0, chunk, TILE)]
    assert all(p["mode"] == 1 and p["k"] >= 2 for p in plans)
    assert sum(p["n_esc"] for p in plans) > 65535
    payload = oracle.encode(0, state, chunk)
    v, staging, _ = oracle.decode_verify(0, payload, state.size, chunk)
    assert v == 0 and np.array_equal(staging[:state.size], state)


def test_payload_bound_counts_tiles():
    raw = 16 + 2 * 32768  # a RAW record of a full tile
    for chunk in (1 << 17, 1 << 22, 1 << 24):
        per = chunk // TILE
        for n in (0, 1, 7):
            assert oracle.payload_bound(123, chunk, n) == 64 + n * per * (16 + raw)
    # at most 64 KiB the unit is the chunk
    assert oracle.payload_bound(123, 4096, 3) == 64 + 3 * (16 + 16 + 2 * 2048)
