"""GPU parity: every libwm output equals the oracle's, bit for bit.

Runs through the C ABI (ctypes) on device buffers; the oracle runs on host
copies of the same bytes.  Checksums, dirty lists, payload bytes, decoded
bytes and verdicts are compared exactly (integer work: tolerance 0).
"""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

pytestmark = pytest.mark.gpu

CH = 65536


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def mover(nbytes, kind=0, **kw):
    from paper_2607_10389_amd import Mover
    return Mover(nbytes, kind, **kw)


from gpu_helpers import (ORACLE_THREADS, check_full_ship, host_bytes,  # noqa: E402
                         random_bytes, say, u32)


@pytest.mark.parametrize("kind", [0, 1])
def test_tiny_checksum(wm, kind):
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    m = mover(state.numel() * 2, kind)
    m.checksum(state)
    torch.cuda.synchronize()
    crcs, g = oracle.checksum_chunks(kind, host_bytes(state), CH)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g


@pytest.mark.parametrize("n", [1, 15, 16, 17, 4095, 65535, 65536, 65537,
                               2 * CH + 5536, 5 * CH + 1, 7 * CH - 2])
def test_ragged_checksum(wm, n):
    say(f"[ragged checksum] n={n}")
    data = random_bytes(n, seed=n)
    m = mover(n)
    m.checksum(data)
    torch.cuda.synchronize()
    crcs, g = oracle.checksum_chunks(0, host_bytes(data), CH)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g


# The global CRC folds the n - 1 full chunks' CRCs in runs of four, 4096
# pieces per pass over the workgroup (zeros padded in front): these counts
# sit on either side of one and two passes.
@pytest.mark.parametrize("chunks,tail", [(4096, CH), (4097, CH), (4098, 777),
                                         (8193, CH), (8194, 3)])
def test_global_crc_fold_boundaries(wm, chunks, tail):
    n = (chunks - 1) * CH + tail
    say(f"[fold boundaries] chunks={chunks} tail={tail}")
    data = random_bytes(n, seed=chunks)
    kind = chunks & 1
    m = mover(n, kind)
    m.checksum(data)
    torch.cuda.synchronize()
    crcs, g = oracle.checksum_chunks(kind, host_bytes(data), CH, ORACLE_THREADS)
    assert np.array_equal(m.crc_host(), crcs)
    assert int(u32(m.global_crc)[0]) == g


def test_full_ship_at_a_fold_boundary(wm):
    """4098 chunks (the last one short) of bf16 values: the global CRC and
    the table CRC (4098 entries) both take two passes of the fold."""
    n_words = (4097 * CH + 778) // 2
    gen = torch.Generator(device="cuda").manual_seed(4098)
    state = torch.randn(n_words, generator=gen, device="cuda").to(torch.bfloat16)
    m = mover(n_words * 2)
    check_full_ship(m, state, 0, "fold boundary")


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("fused", [True, False])
def test_tiny_full_ship(wm, kind, fused):
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    m = mover(state.numel() * 2, kind)
    check_full_ship(m, state, kind, "tiny", fused)


@pytest.mark.parametrize("codec", [1, 2])
def test_invalid_index_list_gives_an_empty_payload(wm, codec):
    """A list that repeats, goes backwards or leaves the chunk range is
    rejected on the device (empty payload); a valid list on the same
    buffers afterwards encodes exactly as the oracle does."""
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    nbytes = state.numel() * 2
    m = mover(nbytes, 0, codec=codec)
    m.checksum(state)
    # the last list is one entry longer than the chunk count: its first 32
    # entries alone would be a valid full list
    for bad in ([3, 3, 5], [5, 2, 9], [0, 1, 32], [7, 40], list(range(32)) + [32]):
        idx = torch.tensor(bad, dtype=torch.int32, device="cuda")
        n_idx = torch.tensor([len(bad)], dtype=torch.int32, device="cuda")
        m.payload_bytes.fill_(123)
        m.payload[:64].fill_(0xEE)
        wm.encode(state, nbytes, m.p, idx, n_idx, m.crc, m.payload, m.payload_bytes, m.ws_src)
        torch.cuda.synchronize()
        assert int(m.payload_bytes.item()) == 0, (codec, bad)
        assert not m.payload[:64].any(), (codec, bad)
    good = np.array([1, 4, 9, 31], dtype=np.uint32)
    idx = torch.from_numpy(good.view(np.int32)).cuda()
    n_idx = torch.tensor([good.size], dtype=torch.int32, device="cuda")
    wm.encode(state, nbytes, m.p, idx, n_idx, m.crc, m.payload, m.payload_bytes, m.ws_src)
    torch.cuda.synchronize()
    want = oracle.encode(0, host_bytes(state), CH, good, ORACLE_THREADS, codec=codec)
    assert np.array_equal(m.payload_host(), want)


def test_tiny_full_ship_crc_in_pass(wm):
    """wm_encode with crc = NULL computes the receipts in the same pass."""
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    m = mover(state.numel() * 2)
    m.encode(state, with_crc=False)
    torch.cuda.synchronize()
    want = oracle.encode(0, host_bytes(state), CH)
    assert np.array_equal(m.payload_host(), want)


def test_tiny_step(wm):
    prev, cur, ids = wm_inputs.tiny_step("cuda")
    nbytes = cur.numel() * 2
    hc, hp = host_bytes(cur), host_bytes(prev)
    want_idx = oracle.diff_dirty(hc, hp, CH)
    assert want_idx.tolist() == ids.cpu().tolist()
    crcs, _ = oracle.checksum_chunks(0, hc, CH)
    want_payload = oracle.encode(0, hc, CH, want_idx)

    # separate calls
    m = mover(nbytes)
    m.checksum(cur)
    m.diff(cur, prev)
    m.encode(cur, dirty_only=True)
    torch.cuda.synchronize()
    assert np.array_equal(m.dirty_host(), want_idx)
    assert np.array_equal(m.crc_host(), crcs)
    assert np.array_equal(m.payload_host(), want_payload)

    # fused step
    m2 = mover(nbytes)
    m2.encode_step(cur, prev)
    torch.cuda.synchronize()
    assert np.array_equal(m2.dirty_host(), want_idx)
    assert np.array_equal(m2.crc_host(), crcs)
    assert np.array_equal(m2.payload_host(), want_payload)

    # destination: decode into compact staging, scatter-install into live
    live = prev.clone()
    m2.decode()
    assert m2.commit(live, scatter=True) == 0
    assert torch.equal(live, cur)
    v, staging, _ = oracle.decode_verify(0, want_payload, nbytes, CH)
    assert v == 0
    n = want_idx.size
    assert np.array_equal(host_bytes(m2.staging[: n * CH]), staging[: n * CH])


def _words_state(words: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(words.astype(np.uint16).view(np.int16).copy()).cuda()


def edge_states():
    rng = np.random.default_rng(17)
    n = CH // 2
    yield "constant", np.full(3 * n, 0x3F80)
    yield "random_bits", rng.integers(0, 65536, 3 * n)
    yield "all_patterns", np.arange(65536 * 2) % 65536
    yield "special", np.resize(np.array([0x7FC0, 0x7F81, 0xFFC1, 0x7F80, 0xFF80,
                                         0, 0x8000, 1, 0x807F, 0x7F7F]), 2 * n)
    t = (rng.standard_t(3, 4 * n) * 10).astype(np.float32)
    yield "student_t", (t.view(np.uint32) >> 16)
    x = rng.standard_normal(3 * n + 2768).astype(np.float32)
    yield "ragged_tail", (x.view(np.uint32) >> 16)
    wide = np.concatenate([rng.integers(0, 256, 16) << 7, np.full(n - 16, 127 << 7)])
    yield "few_escapes", wide
    yield "top_exponents", (np.resize([254, 255, 253], n) << 7) | rng.integers(0, 128, n)
    yield "one_word_tail", np.concatenate([np.full(n, 0x4000), [0x1234]])


@pytest.mark.parametrize("label,words", list(edge_states()),
                         ids=[s[0] for s in edge_states()])
def test_codec_edge_cases(wm, label, words):
    state = _words_state(np.asarray(words))
    m = mover(state.numel() * 2)
    check_full_ship(m, state, 0, label, fused=True)


def test_empty_state(wm):
    from paper_2607_10389_amd import _wm
    m = mover(0)
    state = torch.zeros(16, dtype=torch.uint8, device="cuda")
    m.encode_step(state, None)
    torch.cuda.synchronize()
    want = oracle.encode(0, np.zeros(0, np.uint8), CH)
    assert np.array_equal(m.payload_host(), want)
    m.decode()
    assert m.commit(None, scatter=False) == _wm.WM_OK


def test_bit_flips_abort_and_match_oracle(wm):
    """Flipped payload bits: the GPU verdict equals the oracle's, and a
    scatter commit after a nonzero verdict leaves live untouched."""
    rng = np.random.default_rng(4)
    n = CH // 2
    x = rng.standard_normal(n).astype(np.float32)
    words = np.concatenate([x.view(np.uint32) >> 16, rng.integers(0, 65536, n),
                            np.full(700, 0xBF80)])
    state = _words_state(words)
    nbytes = state.numel() * 2
    m = mover(nbytes)
    m.encode_step(state, None)
    torch.cuda.synchronize()
    good = m.payload_host()
    assert np.array_equal(good, oracle.encode(0, host_bytes(state), CH))
    n_rec = 3
    table = good.size - 16 * n_rec
    positions = list(range(0, 64)) + list(range(64, 64 + 16)) + \
        list(range(table, good.size)) + \
        rng.integers(0, good.size, 120).tolist()
    live0 = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    for pos in positions:
        bit = int(rng.integers(0, 8))
        bad = good.copy()
        bad[pos] ^= 1 << bit
        m.payload[: bad.size].copy_(torch.from_numpy(bad))
        m.decode(payload_cap=bad.size)
        live = live0.clone()
        rc = m.commit(live, scatter=True)
        v_gpu = int(m.verdict.item())
        v_orc, _, st = oracle.decode_verify(0, bad, nbytes, CH)
        assert v_orc != 0 and v_gpu == v_orc, (pos, bit, v_gpu, v_orc)
        assert rc == 1
        assert not live.any()
        if v_orc & (oracle.V_RECORD | oracle.V_DATA):
            assert np.array_equal(u32(m.rec_status)[:n_rec], st[:n_rec]), pos


def test_truncation_and_wrong_params(wm):
    from paper_2607_10389_amd import _wm
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    nbytes = state.numel() * 2
    m = mover(nbytes)
    m.encode_step(state, None)
    size = int(m.payload_bytes.item())
    m.decode(payload_cap=size - 16)
    assert m.commit(None, scatter=False) == _wm.WM_VERIFY_FAILED
    assert int(m.verdict.item()) == oracle.V_HEADER
    # receiver expecting another size
    m2 = mover(nbytes - 2)
    m2.decode(payload=m.payload, payload_cap=size)
    assert m2.commit(None, scatter=False) == _wm.WM_VERIFY_FAILED
    # staging too small
    m3 = mover(nbytes, staging_chunks=4)
    m3.decode(payload=m.payload, payload_cap=size)
    assert m3.commit(None, scatter=False) == _wm.WM_VERIFY_FAILED
    assert int(m3.verdict.item()) == oracle.V_STAGING


def test_production_full_ship(wm):
    state = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    say("[production] generated")
    m = mover(state.numel() * 2)
    got = check_full_ship(m, state, 0, "production", fused=True)
    say(f"[production] payload {got.size} bytes, ratio {got.size / (state.numel() * 2):.4f}")


def _exp_words(rng, n, width, base, esc_frac):
    """n bf16 words whose exponents are uniform over [base, base + width),
    a fraction esc_frac of them replaced by uniform exponents over 0..255;
    sign and mantissa uniform."""
    e = base + rng.integers(0, width, n)
    m = rng.random(n) < esc_frac
    e[m] = rng.integers(0, 256, int(m.sum()))
    sm = rng.integers(0, 256, n)
    return ((sm >> 7) << 15) | (e << 7) | (sm & 127)


def code_width_state(k: int) -> np.ndarray:
    """Three chunks whose oracle plan is PACK with code width k: a full chunk
    with 2% escapes, a full chunk with none (5% escapes for k = 1, where a
    window of one exponent and no escapes is the constant record), and a
    5,536-byte tail with 2% escapes."""
    rng = np.random.default_rng(100 + k)
    width = (1 << k) - 1
    base = 128 - width // 2
    n = CH // 2
    return np.concatenate([_exp_words(rng, n, width, base, 0.02),
                           _exp_words(rng, n, width, base, 0.05 if k == 1 else 0.0),
                           _exp_words(rng, 2768, width, base, 0.02)]).astype(np.uint16)


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("k", range(1, 8))
def test_every_code_width(wm, k, kind):
    """PACK records of every code width k = 1..7 (the k-specialised packing
    and unpacking paths, including codes that straddle three dwords for k =
    5..7), on full chunks and a short tail, with and without escapes, through
    the full ship, the encoder with CRCs given, and the fused step."""
    words = code_width_state(k)
    hw = words.view(np.uint8)
    for c in range(3):
        plan = oracle.plan_chunk(hw[c * CH:(c + 1) * CH])
        assert plan["mode"] == 1 and plan["k"] == k, (k, c, plan)
        assert (plan["n_esc"] > 0) == (c != 1 or k == 1), (k, c, plan)
    state = _words_state(words)
    nbytes = state.numel() * 2
    m = mover(nbytes, kind)
    check_full_ship(m, state, kind, f"k={k}", fused=(kind == 0))
    # fused step against a snapshot whose chunk 1 is unchanged
    prev = state.clone()
    prev[:10] ^= 1
    prev[-5:] ^= 0x100
    m2 = mover(nbytes, kind)
    m2.encode_step(state, prev)
    torch.cuda.synchronize()
    want_idx = np.array([0, 2], np.uint32)
    assert np.array_equal(m2.dirty_host(), want_idx)
    want = oracle.encode(kind, host_bytes(state), CH, want_idx)
    assert np.array_equal(m2.payload_host(), want), k
    live = prev.clone()
    m2.decode()
    assert m2.commit(live, scatter=True) == 0
    assert torch.equal(live, state)


def test_bit_flips_in_wide_code_records(wm):
    """Flipped bits in PACK k=6 and k=7 records (codes, escape index,
    escapes, sign/mantissa plane, padding): the GPU verdict word and record
    status equal the oracle's, and a scatter commit leaves live untouched."""
    rng = np.random.default_rng(66)
    n = CH // 2
    words = np.concatenate([_exp_words(rng, n, 63, 97, 0.02),
                            _exp_words(rng, 1000, 127, 65, 0.03)]).astype(np.uint16)
    hw = words.view(np.uint8)
    assert oracle.plan_chunk(hw[:CH])["k"] == 6
    assert oracle.plan_chunk(hw[CH:])["k"] == 7
    state = _words_state(words)
    nbytes = state.numel() * 2
    m = mover(nbytes)
    m.encode_step(state, None)
    torch.cuda.synchronize()
    good = m.payload_host()
    assert np.array_equal(good, oracle.encode(0, host_bytes(state), CH))
    n_rec = 2
    positions = rng.integers(64, good.size - 16 * n_rec, 160).tolist()
    live0 = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    for pos in positions:
        bit = int(rng.integers(0, 8))
        bad = good.copy()
        bad[pos] ^= 1 << bit
        m.payload[: bad.size].copy_(torch.from_numpy(bad))
        m.decode(payload_cap=bad.size)
        live = live0.clone()
        rc = m.commit(live, scatter=True)
        v_gpu = int(m.verdict.item())
        v_orc, _, st = oracle.decode_verify(0, bad, nbytes, CH)
        assert v_orc != 0 and v_gpu == v_orc, (pos, bit, v_gpu, v_orc)
        assert rc == 1 and not live.any()
        assert np.array_equal(u32(m.rec_status)[:n_rec], st[:n_rec]), pos


@pytest.mark.parametrize("codec", [1, 2])
def test_list_encode_without_crcs(wm, codec):
    """wm_encode of an index list with crc = NULL: the call checksums every
    chunk itself, so the payload (receipts and the header's global CRC of the
    whole state) equals the oracle's."""
    prev, cur, ids = wm_inputs.tiny_step("cuda")
    nbytes = cur.numel() * 2
    m = mover(nbytes, 1, codec=codec)
    m.diff(cur, prev)
    m.crc.fill_(0x5A5A5A5A)  # not read
    m.encode(cur, dirty_only=True, with_crc=False)
    torch.cuda.synchronize()
    idx = oracle.diff_dirty(host_bytes(cur), host_bytes(prev), CH)
    want = oracle.encode(1, host_bytes(cur), CH, idx, ORACLE_THREADS, codec=codec)
    assert np.array_equal(m.payload_host(), want)
