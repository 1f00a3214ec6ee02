"""Fail-closed pins for the oracle (no GPU).

The paper's contract: the destination is bit-identical to the source or
nothing is installed; commit happens only on a matching fingerprint
(§4 "Sufficiency"; Table 1: migrate stages into a shadow slot, commit or
rollback is the only exit).  Here every single-bit flip of a small payload
must be rejected and must leave `live` untouched, and malformed payloads
(truncation, wrong parameters) must be rejected.
"""
import numpy as np
import pytest

import oracle

CH = 4096


def small_state():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(CH // 2).astype(np.float32)
    packed = (x.view(np.uint32) >> 16).astype(np.uint16).view(np.uint8)
    raw = rng.integers(0, 256, CH, dtype=np.uint8)
    const = np.full(CH // 2, 0xBF80, np.uint16).view(np.uint8)
    return np.concatenate([packed, raw, const[:1000]])  # PACK, RAW, k=0 tail


def test_every_single_bit_flip_aborts():
    state = small_state()
    payload = oracle.encode(0, state, CH)
    plans = [oracle.plan_chunk(state[i:i + CH]) for i in range(0, state.size, CH)]
    assert [p["mode"] for p in plans] == [1, 0, 1]
    assert plans[2]["k"] == 0
    v, _, _ = oracle.decode_verify(0, payload, state.size, CH)
    assert v == 0
    before = np.zeros_like(state)
    for byte in range(payload.size):
        for bit in range(8):
            bad = payload.copy()
            bad[byte] ^= 1 << bit
            v, staging, _ = oracle.decode_verify(0, bad, state.size, CH)
            assert v != 0, (byte, bit)
            live = before.copy()
            assert oracle.commit(live, CH, staging, bad, v) == 1
            assert not live.any()


def test_flip_classes_set_expected_bits():
    state = small_state()
    payload = oracle.encode(0, state, CH)
    n_rec = 3
    rec0 = 64
    table = payload.size - 16 * n_rec

    def verdict_after_flip(pos):
        bad = payload.copy()
        bad[pos] ^= 1
        return oracle.decode_verify(0, bad, state.size, CH)

    assert verdict_after_flip(5)[0] == oracle.V_HEADER
    assert verdict_after_flip(table + 3)[0] == oracle.V_TABLE
    assert verdict_after_flip(rec0 + 1)[0] == oracle.V_RECORD  # record k field
    v, _, st = verdict_after_flip(table - 100)  # sm plane of record 2
    assert v == oracle.V_DATA and st[:3].tolist() == [0, 0, oracle.V_DATA]


def test_truncated_and_mismatched_parameters():
    state = small_state()
    payload = oracle.encode(0, state, CH)
    # truncation: payload_bytes exceeds what was delivered
    assert oracle.decode_verify(0, payload[:-16], state.size, CH)[0] == oracle.V_HEADER
    # wrong expected state size, chunk size, CRC kind
    assert oracle.decode_verify(0, payload, state.size + 2, CH)[0] == oracle.V_HEADER
    assert oracle.decode_verify(0, payload, state.size, 2 * CH)[0] == oracle.V_HEADER
    assert oracle.decode_verify(1, payload, state.size, CH)[0] == oracle.V_HEADER
    # receiver staging too small for the records
    v, _, _ = oracle.decode_verify(0, payload, state.size, CH, staging_cap=CH)
    assert v == oracle.V_STAGING


def test_crc32c_payload_roundtrip_and_flip():
    state = small_state()
    payload = oracle.encode(1, state, CH)
    v, staging, _ = oracle.decode_verify(1, payload, state.size, CH)
    assert v == 0
    live = np.zeros_like(state)
    assert oracle.commit(live, CH, staging, payload, v) == 0
    assert np.array_equal(live, state)
    bad = payload.copy()
    bad[payload.size // 2] ^= 0x10
    assert oracle.decode_verify(1, bad, state.size, CH)[0] != 0


@pytest.mark.parametrize("threads", [1, 4])
def test_diff_matches_brute_force(threads):
    rng = np.random.default_rng(threads)
    n = 13 * CH + 77
    prev = rng.integers(0, 256, n, dtype=np.uint8)
    cur = prev.copy()
    touched = sorted(rng.choice(14, 6, replace=False).tolist())
    for c in touched:
        lo = c * CH
        hi = min(lo + CH, n)
        pos = int(rng.integers(lo, hi))
        cur[pos] ^= 1 + int(rng.integers(0, 255))
    # a chunk rewritten with identical bytes stays clean
    cur[2 * CH:3 * CH] = prev[2 * CH:3 * CH].copy()
    got = oracle.diff_dirty(cur, prev, CH, threads)
    padded = np.zeros(14 * CH, np.uint8)
    pp = padded.copy()
    padded[:n] = cur
    pp[:n] = prev
    brute = np.nonzero((padded.reshape(14, CH) != pp.reshape(14, CH)).any(1))[0]
    assert got.tolist() == brute.tolist()
    assert oracle.diff_dirty(cur, cur, CH, threads).size == 0
