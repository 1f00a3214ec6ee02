"""GPU parity of formats v2 and v3 (codec 2: per-chunk canonical Huffman
codes of the exponent plane in 512 streams; codec 3: the same of the high
byte plane, the bf16 byte-plane split) against the oracle: payload bytes,
decoded bytes, verdict words and record status are equal (tolerance 0) on
the tiny cache, dirty lists, edge-case states, flipped bits and the
production-size cache."""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

from gpu_helpers import ORACLE_THREADS, host_bytes, random_bytes, say, u32

pytestmark = pytest.mark.gpu

CH = 65536


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


@pytest.fixture(params=[2, 3], ids=["v2", "v3"])
def codec(request):
    return request.param


def mover(nbytes, kind=0, codec=2):
    from paper_2607_10389_amd import Mover
    return Mover(nbytes, kind, codec=codec)


def dev(a: np.ndarray) -> torch.Tensor:
    t = torch.empty(max(a.size, 16), dtype=torch.uint8, device="cuda")
    t[: a.size] = torch.from_numpy(a).cuda()
    return t


def ship(wm, state_h: np.ndarray, kind=0, label="", codec=2):
    """Full v2 ship of a host state through the GPU; checks payload, decode
    and verdict against the oracle.  Returns the payload."""
    st = dev(state_h)
    m = mover(state_h.size, kind, codec)
    m.encode(st, with_crc=False)
    torch.cuda.synchronize()
    got = m.payload_host()
    want = oracle.encode(kind, state_h, CH, None, ORACLE_THREADS, codec=codec)
    assert got.size == want.size, (label, got.size, want.size)
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: {bad.size} payload bytes differ, first {bad[:8].tolist()}")
    m.decode()
    assert m.commit(None, scatter=False) == wm.WM_OK, label
    torch.cuda.synchronize()
    assert np.array_equal(m.staging[: state_h.size].cpu().numpy(), state_h), label
    return got, m


@pytest.mark.parametrize("kind", [0, 1])
def test_tiny_full_ship(wm, kind, codec):
    state = host_bytes(wm_inputs.make_cache(wm_inputs.TINY))
    got, _ = ship(wm, state, kind, f"tiny kind={kind}", codec)
    say(f"[v{codec}] tiny ratio {got.size / state.size:.4f}")


def _edge_states():
    rng = np.random.default_rng(7)
    n = 3 * CH // 2
    out = {}
    out["constant"] = np.full(n, 0x3F80, np.uint16).view(np.uint8)
    out["random_bits"] = rng.integers(0, 1 << 16, n, dtype=np.uint16).view(np.uint8)
    out["all_patterns"] = np.arange(1 << 16, dtype=np.uint16).view(np.uint8).copy()
    sp = np.array([0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC1, 0x0001, 0x8001, 0x3F80], np.uint16)
    out["special"] = sp[rng.integers(0, sp.size, n)].view(np.uint8)
    t = (rng.standard_t(3, n) * 10).astype(np.float32)
    out["student_t"] = (t.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    x = (rng.standard_normal(n) * 2).astype(np.float32)
    bf = (x.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    out["tail_5536"] = bf[: 2 * CH + 5536].copy()
    out["tail_4098"] = bf[: 2 * CH + 4098].copy()  # a row piece straddles the end
    out["one_word_tail"] = bf[: CH + 2].copy()
    out["two_exponents"] = np.where(rng.random(n) < 0.9, 0x3F80, 0x4000).astype(np.uint16).view(np.uint8)
    # more than 64 distinct exponents in a chunk that still codes as HUF (the
    # plan's code construction past one wave's 64 lanes, and the length cap)
    for scale in (6, 20):
        e = np.clip(127 + np.round(rng.laplace(0, scale, n)), 0, 255).astype(np.int64)
        sm = rng.integers(0, 256, n)
        w = (((sm >> 7) << 15) | (e << 7) | (sm & 127)).astype(np.uint16)
        out[f"laplace_{scale}"] = w.view(np.uint8)
    # exactly 64 and 65 distinct exponents in every chunk, with geometric
    # counts (codes past the length cap, several capping passes): the two
    # sides of the 64-symbol limit of the register-resident construction
    rng2 = np.random.default_rng(11)
    for m_sym in (64, 65):
        g = np.minimum(rng2.geometric(0.12, n) - 1, m_sym - 1)
        for cw in range(0, n, CH // 2):
            g[cw:cw + m_sym] = np.arange(m_sym)
        e = 60 + g
        sm = rng2.integers(0, 256, n)
        w = (((sm >> 7) << 15) | (e << 7) | (sm & 127)).astype(np.uint16)
        out[f"exact_{m_sym}_exponents"] = w.view(np.uint8)
    return out


@pytest.mark.parametrize("scale,min_distinct", [(6, 100), (20, 240)])
def test_wide_alphabet_states_plan_huf(scale, min_distinct):
    """The wide-alphabet edge states really have more than 64 symbols per
    chunk and plan HUF (so the GPU test of them exercises that path)."""
    state = _edge_states()[f"laplace_{scale}"]
    for c in range(0, state.size, CH):
        ch = state[c:c + CH]
        e = (ch.view(np.uint16) >> 7) & 255
        assert np.unique(e).size >= min_distinct
        plan = oracle.plan_chunk_v2(ch)
        assert plan["mode"] == 2 and plan["k"] == 11, plan


@pytest.mark.parametrize("m_sym", [64, 65])
def test_boundary_alphabet_states_plan_huf(m_sym):
    """The boundary states have exactly 64 or 65 exponents in every chunk
    and plan HUF at the length cap (so their GPU test exercises both sides
    of the 64-symbol limit, with capping passes)."""
    state = _edge_states()[f"exact_{m_sym}_exponents"]
    for c in range(0, state.size, CH):
        ch = state[c:c + CH]
        assert np.unique((ch.view(np.uint16) >> 7) & 255).size == m_sym
        plan = oracle.plan_chunk_v2(ch)
        assert plan["mode"] == 2 and plan["k"] == 11, plan


@pytest.mark.parametrize("name", list(_edge_states().keys()))
def test_edge_cases(wm, name, codec):
    state = _edge_states()[name]
    got, _ = ship(wm, state, 0, name, codec)
    modes = got[64]
    say(f"[v{codec}] {name}: {state.size} B -> {got.size} B, first record mode {modes}")


def test_empty_state(wm, codec):
    m = mover(0, 0, codec)
    state = torch.zeros(16, dtype=torch.uint8, device="cuda")
    m.encode(state, with_crc=False)
    torch.cuda.synchronize()
    want = oracle.encode(0, np.zeros(0, np.uint8), CH, None, 1, codec=codec)
    assert np.array_equal(m.payload_host(), want)
    m.decode()
    assert m.commit(None, scatter=False) == wm.WM_OK


def test_dirty_list(wm, codec):
    prev, cur, ids = wm_inputs.tiny_step("cuda")
    h = host_bytes(cur)
    m = mover(h.size, 0, codec)
    m.checksum(cur)
    m.diff(cur, prev)
    m.encode(cur, dirty_only=True)
    torch.cuda.synchronize()
    idx = m.dirty_host()
    want = oracle.encode(0, h, CH, idx, ORACLE_THREADS, codec=codec)
    assert np.array_equal(m.payload_host(), want)
    live = prev.clone().view(-1).view(torch.uint8)
    m.decode()
    assert m.commit(live, scatter=True) == wm.WM_OK
    torch.cuda.synchronize()
    assert torch.equal(live, cur.view(-1).view(torch.uint8))


def test_bit_flips_match_oracle(wm, codec):
    state = _edge_states()["tail_4098"]
    good, m = ship(wm, state, 0, "flips", codec)
    n_rec = int(good[24:28].view(np.uint32)[0])
    total = int(good[32:40].view(np.uint64)[0])
    table = total - 16 * n_rec
    rng = np.random.default_rng(11)
    # header, table, every record's header, tables, streams and planes
    positions = [3, 30, 45, 61, table + 5, table + 16 * (n_rec - 1) + 9]
    positions += list(rng.integers(64, table, 40))
    for pos in positions:
        for bit in (0, 5):
            bad = good.copy()
            bad[pos] ^= 1 << bit
            m.payload[: bad.size] = torch.from_numpy(bad).cuda()
            m.decode()
            torch.cuda.synchronize()
            v = int(m.verdict.item())
            v_o, _, rs_o = oracle.decode_verify(0, bad, state.size, CH, m.staging.numel(),
                                                ORACLE_THREADS, codec=codec)
            assert v == v_o and v != 0, (pos, bit, v, v_o)
            if v_o & 3 == 0:
                assert np.array_equal(u32(m.rec_status)[:n_rec], rs_o[:n_rec]), (pos, bit)


def test_production_full_ship(wm, codec):
    state = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    nbytes = state.numel() * 2
    m = mover(nbytes, 0, codec)
    m.checksum(state)
    m.encode(state)
    torch.cuda.synchronize()
    got = m.payload_host()
    h = host_bytes(state)
    want = oracle.encode(0, h, CH, None, ORACLE_THREADS, codec=codec)
    assert got.size == want.size
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{bad.size} bytes differ, first {bad[:8].tolist()}")
    say(f"[v{codec}] production ratio {got.size / nbytes:.5f}")
    del want, h
    m.decode()
    assert m.commit(None, scatter=False) == wm.WM_OK
    torch.cuda.synchronize()
    assert torch.equal(m.staging[:nbytes], state.view(-1).view(torch.uint8))


def test_huf_record_longer_than_raw_is_rejected(wm, codec):
    from test_oracle_codec_v2 import _huf_payload
    from test_oracle_codec_v3 import _payload
    rng = np.random.default_rng(13)
    st = rng.integers(0, 1 << 16, 3000, dtype=np.uint16).view(np.uint8)
    p = np.frombuffer(_huf_payload(st) if codec == 2 else _payload(st, True), np.uint8)
    m = mover(st.size, 0, codec)
    m.payload[: p.size] = torch.from_numpy(p.copy()).cuda()
    m.decode()
    torch.cuda.synchronize()
    assert int(m.verdict.item()) == 4
    assert int(u32(m.rec_status)[0]) == 4


@pytest.mark.parametrize("kind", [0, 1])
def test_v2_encode_step(wm, kind, codec):
    """Format v2 through the fused call: full ship and the tiny 75%-dirty
    step give the oracle's CRCs, global CRC, dirty list and payload, and the
    step's scatter install leaves live equal to the source."""
    prev, cur, ids = wm_inputs.tiny_step("cuda")
    hc, hp = host_bytes(cur), host_bytes(prev)
    n = hc.size
    m = mover(n, kind, codec)
    m.encode_step(cur, None)
    torch.cuda.synchronize()
    assert np.array_equal(m.payload_host(), oracle.encode(kind, hc, CH, None, 1, codec=codec))
    assert np.array_equal(m.dirty_host(), np.arange(n // CH, dtype=np.uint32))
    crcs, g = oracle.checksum_chunks(kind, hc, CH)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g
    m.encode_step(cur, prev)
    torch.cuda.synchronize()
    idx = oracle.diff_dirty(hc, hp, CH)
    assert np.array_equal(m.dirty_host(), idx)
    assert np.array_equal(m.crc_host(), crcs)
    assert np.array_equal(m.payload_host(), oracle.encode(kind, hc, CH, idx, 1, codec=codec))
    live = prev.clone()
    m.decode()
    assert m.commit(live, scatter=True) == wm.WM_OK
    assert torch.equal(live, cur)
    # no dirty_idx, n_dirty or crc_out from the caller: the workspace holds them
    m2 = mover(n, kind, codec)
    wm.encode_step(cur, prev, n, m2.p, None, None, None, None, m2.payload, m2.payload_bytes,
                   m2.ws_src)
    torch.cuda.synchronize()
    assert np.array_equal(m2.payload_host(), m.payload_host())


@pytest.mark.parametrize("batch", [0, 200_000, 1 << 40])
def test_v2_pipelined_receive(wm, batch, codec):
    """Format v2 received in record batches: verdict, record status and
    staging equal the oracle's decode of the same bytes, also with a flipped
    bit in a record and in the table."""
    prev, cur, _ = wm_inputs.tiny_step("cuda")
    hc, hp = host_bytes(cur), host_bytes(prev)
    idx = oracle.diff_dirty(hc, hp, CH)
    good = oracle.encode(0, hc, CH, idx, 1, codec=codec)
    n = hc.size
    m = mover(n, 0, codec)
    for label, flip in (("clean", None), ("record", 64 + 300), ("table", good.size - 20)):
        bad = good.copy()
        if flip is not None:
            bad[flip] ^= 0x10
        host = torch.empty(bad.size, dtype=torch.uint8, pin_memory=True)
        host[:] = torch.from_numpy(bad)
        cs = torch.cuda.Stream()
        m.payload.fill_(0xA7)
        torch.cuda.synchronize()
        m.receive(host, bad.size, batch, cs)
        torch.cuda.synchronize()
        v = int(m.verdict.item())
        v_o, st_o, rs_o = oracle.decode_verify(0, bad, n, CH, m.staging.numel(), 1, codec=codec)
        assert v == v_o, (label, v, v_o)
        if v_o & 3 == 0:
            k = idx.size
            assert np.array_equal(u32(m.rec_status)[:k], rs_o[:k]), label
        if v_o == 0:
            got = m.staging[: idx.size * CH].cpu().numpy()
            assert np.array_equal(got, st_o[: idx.size * CH]), label
        else:
            assert flip is not None


def test_v2_precopy_rounds(wm, codec):
    """Pre-copy rounds in format v2: each round's dirty list and payload
    equal the oracle's, and the destination ends equal to the source."""
    spec = wm_inputs.TINY
    cur = wm_inputs.make_cache(spec, "cuda")
    n = spec.nbytes
    shipped = torch.zeros(n, dtype=torch.uint8, device="cuda")
    dest = torch.zeros_like(shipped)
    m = mover(n, 0, codec)
    for k in range(4):
        cur_h, shp_h = host_bytes(cur), shipped.cpu().numpy()
        st, nd = m.precopy_round(cur, shipped, dest)
        assert st == wm.WM_OK, k
        got = m.dirty_host()
        assert np.array_equal(got, oracle.diff_dirty(cur_h, shp_h, CH)), k
        assert np.array_equal(m.payload_host(), oracle.encode(0, cur_h, CH, got, 1, codec=codec)), k
        crcs, g = oracle.checksum_chunks(0, cur_h, CH)
        assert np.array_equal(m.crc_host(), crcs), k
        assert torch.equal(dest, shipped)
        writes = wm_inputs.chunk_writes(n // CH, 9, seed=70 + k, device="cuda")
        wm_inputs.rewrite_chunks(cur, spec, writes, seed=80 + k)
    st, nd = m.precopy_round(cur, shipped, dest)
    assert st == wm.WM_OK
    assert torch.equal(dest, cur.view(-1).view(torch.uint8))
