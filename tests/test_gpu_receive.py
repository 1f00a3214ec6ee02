"""GPU parity of the pipelined receive (wm_receive_verify): a payload in
pinned host memory is copied to the device in record batches on a copy
stream while each batch is decoded and verified on the compute stream.  For
every batch size, staging, verdict and record status equal the oracle's
decode of the same bytes, including corrupted and truncated payloads.  The
payloads are the oracle's own encodings (production size: the library's,
which other tests pin to the oracle's)."""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

from gpu_helpers import ORACLE_THREADS, host_bytes, say

pytestmark = pytest.mark.gpu

CH = 65536


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def pinned(a: np.ndarray) -> torch.Tensor:
    t = torch.empty(max(a.size, 1), dtype=torch.uint8, pin_memory=True)
    t[: a.size] = torch.from_numpy(a)
    return t


def receive(m, payload: np.ndarray, batch: int, nbytes_override=None):
    host = pinned(payload)
    cs = torch.cuda.Stream()
    m.payload.fill_(0xA7)  # stale bytes from an earlier move
    torch.cuda.synchronize()
    n = payload.size if nbytes_override is None else nbytes_override
    m.receive(host, n, batch, cs)
    torch.cuda.synchronize()
    return int(m.verdict.item())


def check_against_oracle(m, payload, nbytes, v, label):
    v_o, st_o, rs_o = oracle.decode_verify(0, payload, nbytes, CH, m.staging.numel(),
                                           ORACLE_THREADS)
    assert v == v_o, (label, v, v_o)
    if v_o & 3 == 0:  # header and table valid: per-record status is defined
        n_rec = int(payload[24:28].view(np.uint32)[0])
        got = m.rec_status[:n_rec].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, rs_o[:n_rec]), label
    if v_o == 0:
        n_rec = int(payload[24:28].view(np.uint32)[0])
        got = m.staging[: n_rec * CH].cpu().numpy()
        assert np.array_equal(got, st_o[: n_rec * CH]), label


@pytest.mark.parametrize("batch", [0, 1, 100_000, 300_000, 1 << 40])
def test_full_payload_any_batch(wm, batch):
    from paper_2607_10389_amd import Mover
    state = host_bytes(wm_inputs.make_cache(wm_inputs.TINY))
    payload = oracle.encode(0, state, CH, None, ORACLE_THREADS)
    m = Mover(state.size)
    v = receive(m, payload, batch)
    say(f"[receive] tiny full batch={batch} verdict={v}")
    assert v == 0
    assert np.array_equal(m.staging[: state.size].cpu().numpy(), state)
    check_against_oracle(m, payload, state.size, v, f"batch {batch}")


def test_dirty_payload_with_ragged_tail(wm):
    from paper_2607_10389_amd import Mover
    prev, cur, ids = wm_inputs.tiny_step()
    state = host_bytes(cur)[: 31 * CH + 5536]  # short last chunk
    idx = np.sort(ids.numpy().astype(np.uint32))
    idx = idx[idx < 32]
    payload = oracle.encode(0, state, CH, idx, ORACLE_THREADS)
    m = Mover(state.size)
    v = receive(m, payload, 70_000)
    assert v == 0
    check_against_oracle(m, payload, state.size, v, "dirty")


@pytest.mark.parametrize("where", ["record", "table", "header", "truncated", "garbage"])
def test_corrupted_payloads(wm, where):
    from paper_2607_10389_amd import Mover
    state = host_bytes(wm_inputs.make_cache(wm_inputs.TINY))
    good = oracle.encode(0, state, CH, None, ORACLE_THREADS)
    bad = good.copy()
    n_rec = int(good[24:28].view(np.uint32)[0])
    total = int(good[32:40].view(np.uint64)[0])
    n = bad.size
    if where == "record":
        bad[64 + (total - 64 - 16 * n_rec) // 2] ^= 0x10
    elif where == "table":
        bad[total - 16 * n_rec + 16 * 5 + 9] ^= 1  # an offset of record 5
    elif where == "header":
        bad[24] ^= 2  # record count
    elif where == "truncated":
        n = total - 100
        bad = bad[:n]
    else:
        bad[:64] = 0xEE
    m = Mover(state.size)
    v = receive(m, bad, 100_000, n)
    say(f"[receive] corrupted at {where}: verdict {v}")
    assert v != 0
    check_against_oracle(m, bad[:n], state.size, v, where)


def test_production_payload_in_64mb_batches(wm):
    from paper_2607_10389_amd import Mover
    state = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    nbytes = state.numel() * 2
    src = Mover(nbytes)
    src.encode_step(state, None)
    payload = src.payload_host()
    dst = Mover(nbytes)
    v = receive(dst, payload, 64 << 20)
    say(f"[receive] production payload {payload.size} B in 64 MiB batches: verdict {v}")
    assert v == 0
    assert torch.equal(dst.staging[:nbytes], state.view(-1).view(torch.uint8))
    # the received bytes are the sent bytes
    assert torch.equal(dst.payload[: payload.size].cpu(), torch.from_numpy(payload))


def test_receive_starts_after_earlier_work_on_its_stream(wm):
    """A decode of payload X from the device buffer, then a receive of
    payload Y into the same buffer, enqueued back to back with no host
    synchronisation: the receive's copies wait for the decode, so both
    verify (X's decode never reads Y's bytes)."""
    from paper_2607_10389_amd import Mover
    state = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    nbytes = state.numel() * 2
    src = Mover(nbytes)
    src.encode_step(state, None)
    torch.cuda.synchronize()
    px = int(src.payload_bytes.item())
    dst = Mover(nbytes)
    dst.payload[:px].copy_(src.payload[:px])
    cur, _ = wm_inputs.production_step(state)
    src.encode_step(cur, None)
    y = pinned(src.payload_host())
    v_x = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ds, cs = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    wm.decode_verify(dst.payload, dst.payload.numel(), nbytes, dst.p, dst.staging, v_x,
                     dst.rec_status, dst.ws_dst, ds)
    wm.receive_verify(y, y.numel(), dst.payload, nbytes, dst.p, dst.staging, dst.verdict,
                      dst.rec_status, dst.ws_dst, 64 << 20, cs, ds)
    torch.cuda.synchronize()
    say(f"[receive] after a decode on the same stream: verdicts {int(v_x.item())} "
        f"{int(dst.verdict.item())}")
    assert int(v_x.item()) == 0
    assert int(dst.verdict.item()) == 0
    assert torch.equal(dst.staging[:nbytes], cur.view(-1).view(torch.uint8))
