"""GPU parity at the workload sizes: the active-generation step on the
production-size cache, the eight-session fan-in on eight streams, and the
long-context cache with incompressible chunks and an injected bit flip.

Every byte the C ABI produces (CRCs, dirty lists, payloads, decoded state) is
compared with the oracle on host copies of the same inputs (tolerance 0)."""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

from gpu_helpers import ORACLE_THREADS, host_bytes, say, u32

pytestmark = pytest.mark.gpu

CH = 65536


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def _same(got: np.ndarray, want: np.ndarray, label: str):
    assert got.size == want.size, (label, got.size, want.size)
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: {bad.size} bytes differ, first {bad[:8].tolist()}")


def test_production_active_step(wm):
    """75% of chunks regenerated (Bernoulli, seed 3): fused diff + checksum +
    encode of the dirty chunks, then decode, verify and scatter install."""
    from paper_2607_10389_amd import Mover
    prev = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    cur, ids = wm_inputs.production_step(prev)
    nbytes = cur.numel() * 2
    say(f"[step] {ids.numel()} of {nbytes // CH} chunks regenerated")
    m = Mover(nbytes)
    m.encode_step(cur, prev)
    live = prev.clone()
    torch.cuda.synchronize()
    hc, hp = host_bytes(cur), host_bytes(prev)
    want_idx = oracle.diff_dirty(hc, hp, CH)
    assert np.array_equal(want_idx, ids.cpu().numpy().astype(np.uint32))
    assert np.array_equal(m.dirty_host(), want_idx)
    crcs, g = oracle.checksum_chunks(0, hc, CH, ORACLE_THREADS)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g
    want = oracle.encode(0, hc, CH, want_idx, ORACLE_THREADS)
    _same(m.payload_host(), want, "step payload")
    say("[step] payload matches; decoding")
    m.decode()
    assert m.commit(live, scatter=True) == wm.WM_OK
    torch.cuda.synchronize()
    assert torch.equal(live, cur)


def test_fanin_eight_sessions_on_eight_streams(wm):
    """Eight independent caches encoded and decoded concurrently, one HIP
    stream each (session 7 with CRC-32C)."""
    from paper_2607_10389_amd import Mover
    specs = wm_inputs.FANIN
    states = [wm_inputs.make_cache(s, "cuda") for s in specs]
    streams = [torch.cuda.Stream() for _ in specs]
    kinds = [0] * 7 + [1]
    movers = [Mover(s.numel() * 2, k, stream=st) for s, k, st in zip(states, kinds, streams)]
    torch.cuda.synchronize()
    for m, s, st in zip(movers, states, streams):
        with torch.cuda.stream(st):
            m.encode_step(s, None)
            m.decode()
    torch.cuda.synchronize()
    for i, (m, s, k) in enumerate(zip(movers, states, kinds)):
        h = host_bytes(s)
        _same(m.payload_host(), oracle.encode(k, h, CH, None, ORACLE_THREADS), f"session {i}")
        crcs, g = oracle.checksum_chunks(k, h, CH, ORACLE_THREADS)
        assert np.array_equal(m.crc_host(), crcs), i
        assert int(u32(m.global_crc)[0]) == g, i
        assert int(m.verdict.item()) == 0, i
        assert torch.equal(m.staging[: m.nbytes], s.view(-1).view(torch.uint8)), i
        say(f"[fan-in] session {i} ok")


def _record_modes(payload: np.ndarray) -> np.ndarray:
    n_rec = int(payload[24:28].view(np.uint32)[0])
    total = int(payload[32:40].view(np.uint64)[0])
    table = payload[total - 16 * n_rec: total].view(np.uint64).reshape(n_rec, 2)
    offs = table[:, 1].astype(np.int64)
    return payload[offs]


def test_long_context_raw_chunks_and_bit_flip(wm):
    """4.3 GB Student-t(3) cache with 10% incompressible chunks: the payload
    equals the oracle's (RAW records where the oracle chose them), the
    decoded state equals the source, and one flipped payload bit aborts the
    install with live left untouched."""
    from paper_2607_10389_amd import Mover
    state = wm_inputs.make_cache(wm_inputs.LONG, "cuda")
    nbytes = state.numel() * 2
    say(f"[long] {nbytes} bytes generated")
    m = Mover(nbytes)
    m.encode_step(state, None)
    torch.cuda.synchronize()
    got = m.payload_host()
    h = host_bytes(state)
    want = oracle.encode(0, h, CH, None, ORACLE_THREADS)
    _same(got, want, "long payload")
    modes = _record_modes(got)
    n_raw = int((modes == 0).sum())
    say(f"[long] payload matches; {n_raw} RAW records of {modes.size}")
    assert 0.08 * modes.size < n_raw < 0.12 * modes.size
    del want, h
    m.decode()
    assert m.commit(None, scatter=False) == wm.WM_OK
    assert torch.equal(m.staging[:nbytes], state.view(-1).view(torch.uint8))
    # one bit flipped in the middle of the payload: verify fails, nothing installed
    live = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    pos = got.size // 2 + 12345
    m.payload[pos] ^= 4
    m.decode()
    assert m.commit(live, scatter=True) == wm.WM_VERIFY_FAILED
    torch.cuda.synchronize()
    assert int(m.verdict.item()) != 0
    assert not bool(live.any())
    bad = got.copy()
    bad[pos] ^= 4
    v_orc, _, _ = oracle.decode_verify(0, bad, nbytes, CH, None, ORACLE_THREADS)
    assert int(m.verdict.item()) == v_orc


def test_sessions_on_cu_slices(wm):
    """Two sessions on streams limited to disjoint halves of the CUs (the
    library's grids then span a slice): payloads equal the oracle's and the
    decoded states equal the sources."""
    from paper_2607_10389_amd import Mover, streams
    parts = streams.partition(2)
    try:
        states = [wm_inputs.make_cache(wm_inputs.TINY, "cuda"),
                  wm_inputs.make_cache(wm_inputs.FANIN[1], "cuda")]
        movers = [Mover(s.numel() * 2, 0, stream=p.stream) for s, p in zip(states, parts)]
        torch.cuda.synchronize()
        for m, s in zip(movers, states):
            m.encode_step(s, None)
            m.decode()
        torch.cuda.synchronize()
        for i, (m, s) in enumerate(zip(movers, states)):
            h = host_bytes(s)
            _same(m.payload_host(), oracle.encode(0, h, CH, None, ORACLE_THREADS), f"slice {i}")
            assert m.commit(None, scatter=False) == wm.WM_OK
            assert torch.equal(m.staging[: m.nbytes], s.view(-1).view(torch.uint8)), i
    finally:
        for p in parts:
            p.close()
