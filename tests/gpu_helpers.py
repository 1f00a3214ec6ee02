"""Helpers shared by the GPU parity tests (imported only by `-m gpu` tests)."""
from __future__ import annotations

import os
import sys

import numpy as np
import torch

import oracle

ORACLE_THREADS = min(16, os.cpu_count() or 1)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host_bytes(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(-1).view(torch.uint8).cpu().numpy()


def u32(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


def random_bytes(n: int, seed: int) -> torch.Tensor:
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randint(0, 256, (n,), generator=g, device="cuda",
                         dtype=torch.int32).to(torch.uint8)


def padded(t: torch.Tensor) -> torch.Tensor:
    """Copy into a fresh 256-byte aligned allocation (caching allocator)."""
    out = torch.empty(t.numel(), dtype=t.dtype, device=t.device)
    out.copy_(t)
    return out


def check_full_ship(m, state: torch.Tensor, kind: int, label: str,
                    fused: bool = True):
    """Encode every chunk on the GPU, compare with the oracle, decode, verify
    the decoded bytes.  Returns the host payload."""
    from paper_2607_10389_amd import _wm
    say(f"[{label}] full ship nbytes={m.nbytes} kind={kind} fused={fused}")
    if fused:
        m.encode_step(state, None)
    else:
        m.checksum(state)
        m.encode(state)
    torch.cuda.synchronize()
    host = host_bytes(state)
    want = oracle.encode(kind, host, 65536, None, ORACLE_THREADS)
    got = m.payload_host()
    assert got.size == want.size, (label, got.size, want.size)
    if not np.array_equal(got, want):
        bad = np.nonzero(got != want)[0]
        raise AssertionError(f"{label}: payload differs at {bad.size} bytes, "
                             f"first {bad[:8].tolist()}")
    crcs, g = oracle.checksum_chunks(kind, host, 65536, ORACLE_THREADS)
    assert np.array_equal(m.crc_host(), crcs), label
    assert int(u32(m.global_crc)[0]) == g, label
    m.decode()
    assert m.commit(None, scatter=False) == _wm.WM_OK, label
    torch.cuda.synchronize()
    assert int(m.verdict.item()) == 0, label
    dec = m.staging[: m.nbytes]
    assert torch.equal(dec, state.view(-1).view(torch.uint8)), label
    return got
