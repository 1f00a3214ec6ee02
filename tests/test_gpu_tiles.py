"""GPU parity for chunks above 64 KiB (the paper's pre-copy unit is 4 MB:
§6.2 Exhibit 2, Appendix H).  A chunk stays the unit of dirtiness and of the
per-chunk CRCs; the payload carries one record and one receipt per 64 KiB
tile of each shipped chunk.  Every output (chunk CRCs, global CRC, dirty
chunk lists, payload bytes, verdicts, installed bytes) must equal the
oracle's for the same chunk size, bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

pytestmark = pytest.mark.gpu

TILE = 65536

from gpu_helpers import ORACLE_THREADS, host_bytes, say, u32  # noqa: E402


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def bf16_state(nbytes, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(nbytes // 2, generator=g, device="cuda")
    s = torch.exp(0.5 * torch.randn(1, generator=g, device="cuda"))
    return (x * s).to(torch.bfloat16)


def rewrite_tiles(state, tiles, seed):
    """Copy of state with fresh values in the listed 64 KiB tiles."""
    out = state.clone()
    g = torch.Generator(device="cuda").manual_seed(seed)
    w = TILE // 2
    flat = out.view(-1)
    for t in tiles:
        n = min(w, flat.numel() - t * w)
        flat[t * w:t * w + n] = torch.randn(n, generator=g, device="cuda").to(torch.bfloat16)
    return out


def same(got, want, label):
    assert got.size == want.size, (label, got.size, want.size)
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: {bad.size} bytes differ, first {bad[:8].tolist()}")


def mover(nbytes, kind, chunk, codec=1):
    from paper_2607_10389_amd import Mover
    return Mover(nbytes, kind, chunk_bytes=chunk, codec=codec)


CASES = [(1 << 17, 3 * (1 << 17) + 100_000),  # short last chunk of two tiles
         (1 << 18, 5 * (1 << 18)),             # whole chunks
         (1 << 18, 2 * (1 << 18) + 4 * TILE - 6)]  # last tile short, last chunk 4 tiles


@pytest.mark.parametrize("codec", [1, 2, 3])
@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("chunk,nbytes", CASES)
def test_tiles_full_ship_and_lists(wm, chunk, nbytes, kind, codec):
    say(f"[tiles] chunk={chunk} nbytes={nbytes} kind={kind} codec={codec}")
    state = bf16_state(nbytes, seed=chunk + nbytes + kind)
    host = host_bytes(state)
    n = -(-nbytes // chunk)
    m = mover(nbytes, kind, chunk, codec)
    # chunk CRCs (folded from tiles on the device) and the global CRC
    m.checksum(state)
    torch.cuda.synchronize()
    crcs, g = oracle.checksum_chunks(kind, host, chunk)
    assert crcs.size == n
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g
    # full ship, with the caller's chunk CRCs and without
    for with_crc in (True, False):
        m.encode(state, dirty_only=False, with_crc=with_crc)
        torch.cuda.synchronize()
        same(m.payload_host(), oracle.encode(kind, host, chunk, None, codec=codec),
             f"full with_crc={with_crc}")
    # chunk lists, with the caller's CRCs and without
    for lst in ([], [1], [0, n - 1], list(range(n))):
        m.dirty_idx[:len(lst)] = torch.tensor(lst, dtype=torch.int32, device="cuda")
        m.n_dirty.fill_(len(lst))
        for with_crc in (True, False):
            m.checksum(state)
            m.encode(state, dirty_only=True, with_crc=with_crc)
            torch.cuda.synchronize()
            want = oracle.encode(kind, host, chunk, np.array(lst, np.uint32), codec=codec)
            same(m.payload_host(), want, f"list {lst} with_crc={with_crc}")
    # decode the last payload (every chunk) and install it into a zero state
    m.decode()
    live = torch.zeros_like(state)
    assert m.commit(live, scatter=True) == wm.WM_OK
    torch.cuda.synchronize()
    assert torch.equal(live, state)


@pytest.mark.parametrize("codec", [1, 2, 3])
@pytest.mark.parametrize("kind", [0, 1])
def test_tiles_step(wm, kind, codec):
    """Dirtiness is the chunk's: a chunk with one rewritten tile ships all of
    its tiles."""
    chunk = 1 << 18
    nbytes = 6 * chunk + 3 * TILE + 2000
    prev = bf16_state(nbytes, seed=40 + kind)
    cur = rewrite_tiles(prev, [1, 8, 9, 23, 26], seed=41)  # chunks 0, 2, 5, 6
    say(f"[tiles step] kind={kind} codec={codec}")
    m = mover(nbytes, kind, chunk, codec)
    m.encode_step(cur, prev)
    torch.cuda.synchronize()
    hc, hp = host_bytes(cur), host_bytes(prev)
    want_idx = oracle.diff_dirty(hc, hp, chunk)
    assert want_idx.tolist() == [0, 2, 5, 6]
    assert np.array_equal(m.dirty_host(), want_idx)
    crcs, g = oracle.checksum_chunks(kind, hc, chunk)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g
    same(m.payload_host(), oracle.encode(kind, hc, chunk, want_idx, codec=codec), "step payload")
    # the separate calls give the same dirty list
    m2 = mover(nbytes, kind, chunk, codec)
    m2.diff(cur, prev)
    torch.cuda.synchronize()
    assert np.array_equal(m2.dirty_host(), want_idx)
    # decode, verify and scatter the dirty tiles into prev
    m.decode()
    live = prev.clone()
    assert m.commit(live, scatter=True) == wm.WM_OK
    torch.cuda.synchronize()
    assert torch.equal(live, cur)
    v, _, st = oracle.decode_verify(kind, m.payload_host(), nbytes, chunk, codec=codec)
    assert v == 0 and int(m.verdict.item()) == 0
    # without prev every chunk ships, the dirty list lists every chunk
    m.encode_step(cur, None)
    torch.cuda.synchronize()
    same(m.payload_host(), oracle.encode(kind, hc, chunk, None, codec=codec), "step full")
    assert np.array_equal(m.dirty_host(), np.arange(-(-nbytes // chunk), dtype=np.uint32))
    assert np.array_equal(m.crc_host(), crcs)


def _rebuilt(kind, payload64, chunk, n):
    """A 64 KiB-chunk payload's bytes with the header's chunk size and count
    set to (chunk, n) and its header CRC recomputed by the oracle's CRC."""
    p = payload64.copy()
    p[8:12] = np.frombuffer(np.uint32(chunk).tobytes(), np.uint8)
    p[12:16] = np.frombuffer(np.uint32(n).tobytes(), np.uint8)
    p[60:64] = np.frombuffer(np.uint32(oracle.crc(kind, p[:60])).tobytes(), np.uint8)
    return p


@pytest.mark.parametrize("codec", [1, 2, 3])
@pytest.mark.parametrize("kind", [0, 1])
def test_tiles_partial_chunk_tables(wm, kind, codec):
    """Tables that ship part of a chunk are table errors; whole chunks pass
    (the verdicts are the oracle's)."""
    chunk = 1 << 18
    nbytes = 2 * chunk + 3 * TILE - 4096
    state = bf16_state(nbytes, seed=7 + kind)
    host = host_bytes(state)
    from paper_2607_10389_amd import _wm
    m = mover(nbytes, kind, chunk, codec)
    cases = [(0, 1, 2, 3), (8, 9, 10), (0, 1, 2, 3, 8, 9, 10), (0, 1, 2), (1, 2, 3),
             (0, 1, 3), (4, 5, 6, 7, 9, 10), (8, 9), (3, 4, 5, 6, 7), (0, 1, 2, 3, 4)]
    for tiles in cases:
        small = oracle.encode(kind, host, TILE, np.array(tiles, np.uint32), codec=codec)
        p = _rebuilt(kind, small, chunk, 3)
        want, _, _ = oracle.decode_verify(kind, p, nbytes, chunk, codec=codec)
        buf = torch.zeros(m.payload.numel(), dtype=torch.uint8, device="cuda")
        buf[:p.size] = torch.from_numpy(p).cuda()
        m.decode(buf)
        torch.cuda.synchronize()
        got = int(m.verdict.item())
        say(f"[tiles table] {tiles}: oracle {want} gpu {got}")
        assert got == want, (tiles, got, want)
        live = torch.zeros_like(state)
        st = m.commit(live, scatter=True, payload=buf)
        assert st == (_wm.WM_OK if want == 0 else _wm.WM_VERIFY_FAILED)
        if want:
            assert int(live.view(torch.int16).abs().sum().item()) == 0


def test_tiles_invalid_lists_give_an_empty_payload(wm):
    chunk = 1 << 17
    nbytes = 4 * chunk
    state = bf16_state(nbytes, seed=3)
    m = mover(nbytes, 0, chunk)
    from paper_2607_10389_amd import _wm
    idx = torch.zeros(8, dtype=torch.int32, device="cuda")
    n_idx = torch.zeros(1, dtype=torch.int32, device="cuda")
    for lst in ([1, 1], [2, 1], [4], [0, 1, 2, 3, 3]):
        idx[:len(lst)] = torch.tensor(lst, dtype=torch.int32, device="cuda")
        n_idx.fill_(len(lst))
        _wm.encode(state, nbytes, m.p, idx, n_idx, None, m.payload, m.payload_bytes, m.ws_src)
        torch.cuda.synchronize()
        assert int(m.payload_bytes.item()) == 0, lst
        assert int(m.payload[:64].abs().sum().item()) == 0, lst
    # then a valid list on the same buffers
    m.dirty_idx[:2] = torch.tensor([0, 3], dtype=torch.int32, device="cuda")
    m.n_dirty.fill_(2)
    m.encode(state, dirty_only=True, with_crc=False)
    torch.cuda.synchronize()
    same(m.payload_host(), oracle.encode(0, host_bytes(state), chunk, np.array([0, 3], np.uint32)),
         "valid list after invalid ones")


def test_tiles_abi_limits(wm):
    from paper_2607_10389_amd import _wm
    nbytes = 1 << 20
    state = bf16_state(nbytes, seed=1)
    # chunks below 64 KiB are valid parameters the kernels do not implement
    p = _wm.params(chunk_bytes=1 << 15)
    assert _wm.workspace_bytes(nbytes, p) == 0
    crc = torch.zeros(32, dtype=torch.int32, device="cuda")
    with pytest.raises(_wm.WmError) as e:
        _wm.checksum_chunks(state, nbytes, p, crc)
    assert e.value.status == _wm.WM_ERR_UNSUPPORTED
    # the built-in workspace has the 64 KiB layout only
    m = mover(nbytes, 0, 1 << 18)
    with pytest.raises(_wm.WmError) as e:
        _wm.encode_step_static(state, None, nbytes, m.p, m.crc, m.global_crc, m.dirty_idx,
                               m.n_dirty, m.payload, m.payload_bytes)
    assert e.value.status == _wm.WM_ERR_UNSUPPORTED


@pytest.mark.parametrize("kind", [0, 1])
def test_tiles_precopy_rounds(wm, kind):
    """Pre-copy rounds in 256 KiB chunks converge to the source; each round's
    dirty list and payload are the oracle's."""
    chunk = 1 << 18
    nbytes = 9 * chunk + 2 * TILE
    src = bf16_state(nbytes, seed=60 + kind)
    shipped = torch.zeros_like(src)
    dest = torch.zeros_like(src)
    m = mover(nbytes, kind, chunk)
    from paper_2607_10389_amd import _wm
    for rnd, tiles in enumerate(([], [3, 17], [36], [])):
        if tiles:
            src = rewrite_tiles(src, tiles, seed=70 + rnd)
        hs, hd = host_bytes(src), host_bytes(shipped)
        want_idx = oracle.diff_dirty(hs, hd, chunk)
        st, nd = m.precopy_round(src, shipped, dest)
        assert st == _wm.WM_OK
        assert nd == want_idx.size
        same(m.payload_host(), oracle.encode(kind, hs, chunk, want_idx), f"round {rnd}")
        assert torch.equal(dest, src) and torch.equal(shipped, src)


@pytest.mark.parametrize("codec", [1, 2, 3])
def test_production_in_4mib_chunks(wm, codec):
    """The production cache is exactly 399 chunks of 4 MiB: full ship and a
    step whose dirty chunks come from the 75% tile rewrite, against the
    oracle in 4 MiB chunks."""
    chunk = 1 << 22
    prev = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    nbytes = prev.numel() * 2
    assert nbytes == 399 * chunk
    hp = host_bytes(prev)
    say(f"[4 MiB] production full ship codec={codec}")
    m = mover(nbytes, 0, chunk, codec)
    m.encode_step(prev, None)
    torch.cuda.synchronize()
    same(m.payload_host(), oracle.encode(0, hp, chunk, None, ORACLE_THREADS, codec=codec),
         "4 MiB full ship")
    crcs, g = oracle.checksum_chunks(0, hp, chunk, ORACLE_THREADS)
    assert np.array_equal(m.crc_host(), crcs) and int(u32(m.global_crc)[0]) == g
    m.decode()
    assert m.commit(None, scatter=False) == 0
    torch.cuda.synchronize()
    assert torch.equal(m.staging[:nbytes], prev.view(-1).view(torch.uint8))
    if codec != 1:
        return
    # a step that rewrites about 2% of the tiles dirties many 4 MiB chunks
    ids = wm_inputs.permuted_chunks(nbytes // TILE, 500, seed=9, device="cuda")
    cur = wm_inputs.regenerate(prev, wm_inputs.PRODUCTION, ids, seed=19)
    hc = host_bytes(cur)
    m.encode_step(cur, prev)
    torch.cuda.synchronize()
    want_idx = oracle.diff_dirty(hc, hp, chunk, ORACLE_THREADS)
    assert np.array_equal(m.dirty_host(), want_idx)
    same(m.payload_host(), oracle.encode(0, hc, chunk, want_idx, ORACLE_THREADS), "4 MiB step")
    m.decode()
    live = prev.clone()
    assert m.commit(live, scatter=True) == 0
    torch.cuda.synchronize()
    assert torch.equal(live, cur)
