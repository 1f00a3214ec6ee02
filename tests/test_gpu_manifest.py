"""GPU parity of the manifest flatten and rehydrate (wm_flatten,
wm_rehydrate) against the oracle: ragged leaves with every edge size, the
450-leaf production manifest, and a move of a manifest end to end (flatten,
encode, decode, verify, install, rehydrate).  Byte work: tolerance 0."""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs

from gpu_helpers import host_bytes, random_bytes, say

pytestmark = pytest.mark.gpu

GUARD = 0x5A


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def carve(sizes, seed):
    """Leaves as views of one device buffer: each at a 256-byte aligned
    offset, followed by guard bytes up to the next leaf."""
    offs, pos = [], 0
    for s in sizes:
        offs.append(pos)
        pos += -(-(s + 48) // 256) * 256
    buf = torch.full((max(pos, 1),), GUARD, dtype=torch.uint8, device="cuda")
    data = random_bytes(max(sum(sizes), 1), seed)
    src = 0
    for o, s in zip(offs, sizes):
        buf[o:o + s] = data[src:src + s]
        src += s
    return buf, [buf[o:o + s] for o, s in zip(offs, sizes)], offs


def guards_intact(buf, offs, sizes):
    mask = torch.ones(buf.numel(), dtype=torch.bool, device="cuda")
    for o, s in zip(offs, sizes):
        mask[o:o + s] = False
    return bool((buf[mask] == GUARD).all())


@pytest.mark.parametrize("n,seed", [(1, 0), (7, 1), (90, 2), (400, 3)])
def test_ragged_leaves(wm, n, seed):
    sizes = wm_inputs.ragged_sizes(n, seed)
    if n == 1:
        sizes = [1_000_003]
    say(f"[manifest] ragged n={n} seed={seed} flat={oracle.flat_layout(sizes)[1]}")
    buf, leaves, offs = carve(sizes, seed)
    total = wm.flat_bytes(leaves)
    assert total == oracle.flat_layout(sizes)[1]
    flat = torch.full((total + 4096,), 0xCC, dtype=torch.uint8, device="cuda")
    ws = torch.empty(wm.manifest_ws_bytes(n), dtype=torch.uint8, device="cuda")
    wm.flatten(leaves, flat, ws)
    torch.cuda.synchronize()
    want = oracle.flatten([host_bytes(x) for x in leaves])
    got = flat.cpu().numpy()
    assert np.array_equal(got[:total], want)
    assert (got[total:] == 0xCC).all()  # bytes past the manifest untouched
    # rehydrate into scrambled leaves from a flat whose gaps hold garbage
    orig = [x.clone() for x in leaves]
    for x in leaves:
        x.fill_(0x33)
    off, _ = oracle.flat_layout(sizes)
    noisy = flat.clone()
    gaps = torch.ones(total, dtype=torch.bool, device="cuda")
    for o, s in zip(off.tolist(), sizes):
        gaps[o:o + s] = False
    noisy[:total][gaps] = 0xEE
    wm.rehydrate(noisy, leaves, ws)
    torch.cuda.synchronize()
    for i, (x, y) in enumerate(zip(leaves, orig)):
        assert torch.equal(x, y), (i, sizes[i])
    assert guards_intact(buf, offs, sizes)


def test_degenerate_manifests(wm):
    flat = torch.full((64,), 0xCC, dtype=torch.uint8, device="cuda")
    ws = torch.empty(wm.manifest_ws_bytes(4), dtype=torch.uint8, device="cuda")
    wm.flatten([], flat, ws)
    empty = [torch.empty(0, dtype=torch.uint8, device="cuda") for _ in range(3)]
    wm.flatten(empty, flat, ws)
    wm.rehydrate(flat, empty, ws)
    one = torch.tensor([7], dtype=torch.uint8, device="cuda")
    wm.flatten(empty + [one], flat, ws)
    torch.cuda.synchronize()
    got = flat.cpu().numpy()
    assert got[0] == 7 and (got[1:16] == 0).all() and (got[16:] == 0xCC).all()


def test_production_manifest(wm):
    """The 450-leaf manifest on the production-size cache (1.67 GB)."""
    leaves = wm_inputs.make_manifest(wm_inputs.PRODUCTION, "cuda")
    assert len(leaves) == 450
    total = wm.flat_bytes(leaves)
    say(f"[manifest] production: {len(leaves)} leaves, {total} flat bytes")
    flat = torch.empty(total, dtype=torch.uint8, device="cuda")
    ws = torch.empty(wm.manifest_ws_bytes(len(leaves)), dtype=torch.uint8, device="cuda")
    wm.flatten(leaves, flat, ws)
    torch.cuda.synchronize()
    want = oracle.flatten([host_bytes(x) for x in leaves])
    got = flat.cpu().numpy()
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"flat differs at {bad.size} bytes, first {bad[:8].tolist()}")
    del want, got
    back = [torch.zeros_like(x) for x in leaves]
    wm.rehydrate(flat, back, ws)
    torch.cuda.synchronize()
    for i, (x, y) in enumerate(zip(back, leaves)):
        assert torch.equal(x, y), i


@pytest.mark.parametrize("kind", [0, 1])
def test_manifest_move_end_to_end(wm, kind):
    """Flatten, encode every chunk, decode with verification, install, and
    rehydrate into fresh tensors: every leaf arrives bit-identical, and the
    receipts equal the oracle's CRCs of the oracle's flat bytes."""
    from paper_2607_10389_amd import Mover
    leaves = wm_inputs.make_manifest(wm_inputs.TINY, "cuda")
    total = wm.flat_bytes(leaves)
    flat = torch.empty(total, dtype=torch.uint8, device="cuda")
    ws = torch.empty(wm.manifest_ws_bytes(len(leaves)), dtype=torch.uint8, device="cuda")
    wm.flatten(leaves, flat, ws)
    m = Mover(total, kind)
    m.encode_step(flat, None)
    m.decode()
    live = torch.zeros(total, dtype=torch.uint8, device="cuda")
    assert m.commit(live, scatter=True) == wm.WM_OK
    back = [torch.empty_like(x) for x in leaves]
    wm.rehydrate(live, back, ws)
    torch.cuda.synchronize()
    want_flat = oracle.flatten([host_bytes(x) for x in leaves])
    crcs, _ = oracle.checksum_chunks(kind, want_flat, 65536)
    assert np.array_equal(m.crc_host(), crcs)
    for i, (x, y) in enumerate(zip(back, leaves)):
        assert torch.equal(x, y), i
