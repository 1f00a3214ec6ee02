"""GPU parity of the re-verifying install (wm_commit_reverify) with the
oracle's: the verdict word and the installed state are equal, on the right
base (installed, equal to the source), on a base that differs in a chunk the
payload does not carry, on staging changed after verification, on a full
ship, with a short last chunk, and on the production-size active step."""
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


def _pair(seed, n_bytes, dirty):
    g = torch.Generator(device="cuda").manual_seed(seed)
    prev = torch.randint(0, 256, (n_bytes,), generator=g, device="cuda",
                         dtype=torch.int32).to(torch.uint8)
    cur = prev.clone()
    for c in dirty:
        lo, hi = c * CH, min((c + 1) * CH, n_bytes)
        cur[lo:hi] = torch.randint(0, 256, (hi - lo,), generator=g, device="cuda",
                                   dtype=torch.int32).to(torch.uint8)
    return prev, cur


def _check(m, live, kind, want_status, label):
    """Run the GPU install and the oracle's on the same bytes."""
    from paper_2607_10389_amd import _wm
    pb = int(m.payload_bytes.item())
    payload = m.payload[:pb].cpu().numpy()
    staging = m.staging.cpu().numpy()
    v0 = int(m.verdict.item())
    host_live = host_bytes(live).copy()
    v_orc = oracle.commit_reverify(kind, host_live, CH, staging, payload, v0)
    st = m.commit_reverify(live)
    torch.cuda.synchronize()
    assert st == want_status, (label, st)
    assert int(m.verdict.item()) == v_orc, (label, int(m.verdict.item()), v_orc)
    assert np.array_equal(host_bytes(live), host_live), label


@pytest.mark.parametrize("kind", [0, 1])
def test_reverify_dirty_ship(wm, kind):
    from paper_2607_10389_amd import Mover
    n = 6 * CH + 1000  # chunk 6 is a 1,000-byte tail
    prev, cur = _pair(11 + kind, n, [1, 4, 6])
    m = Mover(n, kind)
    m.encode_step(cur, prev)
    m.decode()
    torch.cuda.synchronize()
    assert m.dirty_host().tolist() == [1, 4, 6]
    # the right base: installed, bit-identical to the source
    live = prev.clone()
    _check(m, live, kind, wm.WM_OK, "right base")
    assert torch.equal(live, cur)
    # a base differing in a clean chunk: refused, live untouched
    live = prev.clone()
    live[2 * CH + 7] ^= 1
    before = live.clone()
    _check(m, live, kind, wm.WM_VERIFY_FAILED, "other base")
    assert torch.equal(live, before)
    assert int(m.verdict.item()) == wm.V_REVERIFY
    # staging changed after verification: refused
    m.verdict.zero_()
    m.staging[CH + 5] ^= 0x80
    live = prev.clone()
    _check(m, live, kind, wm.WM_VERIFY_FAILED, "stale staging")
    assert torch.equal(live, prev)
    # a failed verification passes through: nothing installed
    m.verdict.fill_(wm.V_DATA)
    live = prev.clone()
    st = m.commit_reverify(live)
    assert st == wm.WM_VERIFY_FAILED and int(m.verdict.item()) == wm.V_DATA
    assert torch.equal(live, prev)


def test_reverify_full_ship_and_empty_dirty_set(wm):
    from paper_2607_10389_amd import Mover
    state = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    n = state.numel() * 2
    m = Mover(n)
    m.encode_step(state, None)
    m.decode()
    live = torch.zeros(n, dtype=torch.uint8, device="cuda")
    _check(m, live, 0, wm.WM_OK, "full ship")
    assert torch.equal(live, state.view(-1).view(torch.uint8))
    # no dirty chunk: installs nothing, and succeeds only on the right base
    m.encode_step(state, state)
    m.decode()
    torch.cuda.synchronize()
    assert int(m.n_dirty.item()) == 0
    live = state.view(-1).view(torch.uint8).clone()
    _check(m, live, 0, wm.WM_OK, "empty, right base")
    live[5] ^= 2
    _check(m, live, 0, wm.WM_VERIFY_FAILED, "empty, other base")


def test_reverify_production_step(wm):
    from paper_2607_10389_amd import Mover
    prev = wm_inputs.make_cache(wm_inputs.PRODUCTION, "cuda")
    cur, ids = wm_inputs.production_step(prev)
    n = prev.numel() * 2
    say(f"[reverify] production step, {ids.numel()} dirty chunks")
    m = Mover(n)
    m.encode_step(cur, prev)
    m.decode()
    live = prev.view(-1).view(torch.uint8).clone()
    assert m.commit_reverify(live) == wm.WM_OK
    assert torch.equal(live, cur.view(-1).view(torch.uint8))
    live = prev.view(-1).view(torch.uint8).clone()
    clean = int(np.setdiff1d(np.arange(n // CH), ids.cpu().numpy())[17])
    live[clean * CH + 100] ^= 1
    before = live.clone()
    assert m.commit_reverify(live) == wm.WM_VERIFY_FAILED
    assert int(m.verdict.item()) == wm.V_REVERIFY
    assert torch.equal(live, before)
