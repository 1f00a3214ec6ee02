"""Pins of the oracle's manifest flatten and rehydrate (§4 "Sufficiency":
the move runs on one flat buffer between a flatten and a rehydrate; §5
"Implementation": a manifest of 450 leaves).  The flat layout is this
project's: leaf i at the sum of the earlier sizes rounded up to 16, zero
bytes in the gaps."""
import numpy as np
import pytest
import torch

import oracle
import wm_inputs


def test_hand_worked_example():
    # leaves of 3, 16, 0 and 1 bytes: offsets 0, 16, 32, 32; 48 flat bytes
    a = np.array([1, 2, 3], np.uint8)
    b = np.arange(100, 116, dtype=np.uint8)
    c = np.zeros(0, np.uint8)
    d = np.array([9], np.uint8)
    off, total = oracle.flat_layout([3, 16, 0, 1])
    assert off.tolist() == [0, 16, 32, 32] and total == 48
    want = bytes([1, 2, 3] + [0] * 13 + list(range(100, 116)) + [9] + [0] * 15)
    assert oracle.flatten([a, b, c, d]).tobytes() == want
    back = oracle.rehydrate(np.frombuffer(want, np.uint8), [3, 16, 0, 1])
    assert [x.tobytes() for x in back] == [a.tobytes(), b.tobytes(), b"", d.tobytes()]


def test_aligned_leaves_concatenate():
    # sizes that are multiples of 16: the flat buffer is plain concatenation
    rng = np.random.default_rng(1)
    leaves = [rng.integers(0, 256, 16 * int(n), dtype=np.uint8)
              for n in rng.integers(0, 300, 40)]
    assert np.array_equal(oracle.flatten(leaves), np.concatenate(leaves))


def test_zero_padding_to_16_leaves_the_flat_unchanged():
    rng = np.random.default_rng(2)
    sizes = wm_inputs.ragged_sizes(60, seed=2)
    leaves = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
    padded = [np.pad(x, (0, -x.size % 16)) for x in leaves]
    flat = oracle.flatten(leaves)
    assert np.array_equal(flat, oracle.flatten(padded))
    assert np.array_equal(flat, np.concatenate(padded))
    # zero-size leaves take no room
    assert np.array_equal(flat, oracle.flatten([x for x in leaves if x.size]))


def test_round_trip_is_identity():
    rng = np.random.default_rng(3)
    sizes = wm_inputs.ragged_sizes(90, seed=3)
    leaves = [rng.integers(0, 256, s, dtype=np.uint8) for s in sizes]
    flat = oracle.flatten(leaves)
    assert flat.size % 16 == 0
    # gap bytes are ignored on the way back
    off, total = oracle.flat_layout(sizes)
    noisy = flat.copy()
    for o, s, o_next in zip(off, sizes, list(off[1:]) + [total]):
        noisy[int(o) + s:int(o_next)] = 0xEE
    back = oracle.rehydrate(noisy, sizes)
    assert all(np.array_equal(x, y) for x, y in zip(back, leaves))


def test_slices_of_one_cache_flatten_to_the_cache():
    # head-group slabs of a contiguous cache, taken in memory order, flatten
    # back to the cache's own bytes (the single-tensor configuration is
    # already flat)
    cache = wm_inputs.make_cache(wm_inputs.TINY)
    L, _, H, _, _ = wm_inputs.TINY.shape
    slabs = []
    for layer in range(L):
        for kv in range(2):
            h0 = 0
            for n in wm_inputs.head_groups(H):
                slabs.append(cache[layer, kv, h0:h0 + n].contiguous().view(torch.int16).numpy())
                h0 += n
    want = cache.view(torch.int16).numpy().reshape(-1).view(np.uint8)
    assert np.array_equal(oracle.flatten(slabs), want)


def test_manifest_structure():
    leaves = wm_inputs.make_manifest(wm_inputs.TINY)
    L, _, H, T, D = wm_inputs.TINY.shape
    n_slab = L * 2 * len(wm_inputs.head_groups(H))
    assert len(leaves) == n_slab + L + wm_inputs.N_CONTROL_LEAVES
    assert sum(x.numel() for x in leaves[:n_slab + L] if x.dtype == torch.bfloat16) \
        == L * 2 * H * T * D
    assert all(x.is_contiguous() for x in leaves)
    # the production manifest has the paper's counts: 420 tensors, 450 leaves
    Lp, _, Hp, _, _ = wm_inputs.PRODUCTION.shape
    assert Lp * 2 * len(wm_inputs.head_groups(Hp)) + Lp == 420
    assert 420 + wm_inputs.N_CONTROL_LEAVES == 450


@pytest.mark.parametrize("sizes", [[], [0], [0, 0, 0], [5], [16, 1, 31]])
def test_degenerate_manifests(sizes):
    leaves = [np.full(s, 7, np.uint8) for s in sizes]
    flat = oracle.flatten(leaves)
    assert flat.size == sum(-(-s // 16) * 16 for s in sizes)
    back = oracle.rehydrate(flat, sizes)
    assert [x.tobytes() for x in back] == [x.tobytes() for x in leaves]
