"""The allocation-free fused source step (wm_encode_step_static) against
wm_encode_step on a caller's workspace: every output byte equal (CRCs,
global CRC, dirty list and count, payload), on two calls in a row where the
second ships a smaller state, so the built-in workspace is reused with
stale contents from the first.  A state beyond the built-in workspace's
65,536 chunks is refused on the host."""
import ctypes

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


def _outputs(wm, nbytes, kind):
    n = max(wm.n_chunks(nbytes), 1)
    i32 = dict(dtype=torch.int32, device="cuda")
    p = wm.params(kind)
    return dict(
        crc=torch.zeros(n, **i32), g=torch.zeros(1, **i32),
        idx=torch.zeros(n, **i32), nd=torch.zeros(1, **i32),
        payload=torch.zeros(wm.payload_bound(nbytes, n, p), dtype=torch.uint8, device="cuda"),
        pb=torch.zeros(1, dtype=torch.int64, device="cuda"))


def _both(wm, cur, prev, kind, label):
    nbytes = cur.numel() * cur.element_size()
    p = wm.params(kind)
    a, b = _outputs(wm, nbytes, kind), _outputs(wm, nbytes, kind)
    # poison the static call's outputs, so nothing passes by being left over
    for t in (b["crc"], b["g"], b["idx"], b["nd"]):
        t.fill_(-1)
    b["payload"].fill_(0xA5)
    ws = torch.zeros(wm.workspace_bytes(nbytes, p), dtype=torch.uint8, device="cuda")
    say(f"[no-alloc] {label}: nbytes={nbytes} prev={'yes' if prev is not None else 'no'}")
    wm.encode_step(cur, prev, nbytes, p, a["crc"], a["g"], a["idx"], a["nd"],
                   a["payload"], a["pb"], ws)
    wm.encode_step_static(cur, prev, nbytes, p, b["crc"], b["g"], b["idx"], b["nd"],
                          b["payload"], b["pb"])
    torch.cuda.synchronize()
    size = int(a["pb"].item())
    assert size > 64 and int(b["pb"].item()) == size, label
    n = wm.n_chunks(nbytes)
    nd = int(a["nd"].item())
    assert int(b["nd"].item()) == nd, label
    assert torch.equal(a["crc"][:n], b["crc"][:n]), label
    assert int(a["g"].item()) == int(b["g"].item()), label
    assert torch.equal(a["idx"][:nd], b["idx"][:nd]), label
    assert torch.equal(a["payload"][:size], b["payload"][:size]), label
    # and both are the oracle's payload
    idx = None if prev is None else u32(b["idx"][:nd])
    want = oracle.encode(kind, host_bytes(cur), CH, idx, ORACLE_THREADS)
    assert np.array_equal(b["payload"][:size].cpu().numpy(), want), label
    return nd


def test_static_workspace_matches_the_caller_workspace(wm):
    # first call: 9 chunks and a ragged tail, 75% of them rewritten
    gen = torch.Generator(device="cuda").manual_seed(5)
    n_words = (8 * CH + 5536) // 2
    prev = torch.randn(n_words, generator=gen, device="cuda").to(torch.bfloat16)
    cur = prev.clone()
    rewrite = torch.randperm(9, generator=gen, device="cuda")[:7]
    for c in rewrite.tolist():
        lo, hi = c * CH // 2, min((c + 1) * CH // 2, n_words)
        cur[lo:hi] = torch.randn(hi - lo, generator=gen, device="cuda").to(torch.bfloat16)
    assert _both(wm, cur, prev, 0, "step, 9 chunks") == 7
    # second call, smaller: the tiny cache's full ship (CRC-32C)
    tiny = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    assert _both(wm, tiny, None, 1, "full ship, tiny") == 32


def test_oversized_state_is_refused_on_the_host(wm):
    """65,537 chunks exceed the built-in workspace: WM_ERR_WORKSPACE, and
    nothing is enqueued (the call returns before touching the buffers)."""
    p = wm.params()
    buf = torch.zeros(64, dtype=torch.uint8, device="cuda")
    nbytes = 65537 * CH
    st = wm.LIB.wm_encode_step_static(
        ctypes.c_void_p(buf.data_ptr()), None, nbytes, ctypes.byref(p), None, None, None,
        None, ctypes.c_void_p(buf.data_ptr()), 1 << 62, ctypes.c_void_p(buf.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert st == wm.WM_ERR_WORKSPACE
    assert not buf.any()
