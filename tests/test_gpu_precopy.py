"""GPU parity of iterative pre-copy (wm_precopy_round and the driver in
paper_2607_10389_amd.precopy) against the oracle: every round's dirty list
equals the oracle's diff of the same bytes and the set of chunks the source
wrote, payloads equal the oracle's encoding, the destination ends
bit-identical, and the per-round dirty counts follow the occupancy law of
App. H (converging below one write per shipped chunk, saturating above)."""
import math

import numpy as np
import pytest
import torch

import oracle
import wm_inputs

from gpu_helpers import ORACLE_THREADS, host_bytes, say

pytestmark = pytest.mark.gpu

CH = 65536
SPEC = wm_inputs.FANIN[0]  # [24,2,8,4096,128] bf16, 402,653,184 B, 6,144 chunks


@pytest.fixture(scope="module")
def wm():
    from paper_2607_10389_amd import _wm
    _wm.init(-1)
    return _wm


def within_law(n_dirty, n, w, sigmas=5.0):
    mean, var = oracle.occupancy_mean(n, w), oracle.occupancy_var(n, w)
    return abs(n_dirty - mean) <= sigmas * math.sqrt(var) + 1


def test_rounds_match_the_oracle_and_the_law(wm):
    from paper_2607_10389_amd import Mover
    cur = wm_inputs.make_cache(SPEC, "cuda")
    nbytes, n = SPEC.nbytes, SPEC.nbytes // CH
    shipped = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dest = torch.zeros_like(shipped)
    m = Mover(nbytes)
    rho, writes = 0.5, None
    for k in range(30):
        cur_h, shp_h = host_bytes(cur), shipped.cpu().numpy()
        st, nd = m.precopy_round(cur, shipped, dest)
        assert st == wm.WM_OK
        got = m.dirty_host()
        assert got.size == nd
        assert np.array_equal(got, oracle.diff_dirty(cur_h, shp_h, CH, ORACLE_THREADS)), k
        if writes is not None:
            # every written chunk got fresh bytes, so the dirty set is the
            # set of chunks written during the previous round
            assert np.array_equal(got, np.unique(writes.cpu().numpy()).astype(np.uint32)), k
            assert within_law(nd, n, writes.numel()), (k, nd, writes.numel())
        # round 0 checksums every chunk; later rounds only the dirty ones
        # and keep the rest: either way the CRCs are those of the state
        crcs, g = oracle.checksum_chunks(0, cur_h, CH, ORACLE_THREADS)
        assert np.array_equal(m.crc_host(), crcs), k
        assert int(m.global_crc.cpu().numpy().view(np.uint32)[0]) == g, k
        if k in (0, 1) or nd <= 8:
            want = oracle.encode(0, cur_h, CH, got, ORACLE_THREADS)
            assert np.array_equal(m.payload_host(), want), k
        assert torch.equal(dest, shipped)
        say(f"[precopy] round {k}: {nd} dirty")
        if nd <= 8:
            break
        w = int(round(rho * nd))
        writes = wm_inputs.chunk_writes(n, w, seed=1000 + k, device="cuda")
        wm_inputs.rewrite_chunks(cur, SPEC, writes, seed=2000 + k)
    else:
        raise AssertionError("pre-copy did not converge at 0.5 writes per shipped chunk")
    assert torch.equal(dest, cur.view(-1).view(torch.uint8))


def test_driver_saturates_above_one_write_per_chunk(wm):
    from paper_2607_10389_amd import Mover, precopy
    cur = wm_inputs.make_cache(SPEC, "cuda")
    nbytes, n = SPEC.nbytes, SPEC.nbytes // CH
    shipped = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dest = torch.zeros_like(shipped)
    m = Mover(nbytes)
    rho = 1.93

    def write(k, nd):
        ids = wm_inputs.chunk_writes(n, int(round(rho * nd)), seed=3000 + k, device="cuda")
        wm_inputs.rewrite_chunks(cur, SPEC, ids, seed=4000 + k)

    rounds = precopy.run(m, cur, shipped, dest, write, stop_chunks=0, max_rounds=8)
    fr = [r["dirty"] / n for r in rounds]
    say(f"[precopy] saturating dirty fractions {[round(f, 4) for f in fr]}")
    assert len(rounds) == 9 and rounds[-1]["live"] is False
    pred = oracle.precopy_recursion(n, rho, rounds[0]["dirty"], 8)
    for r, p in zip(rounds[3:8], pred[3:8]):
        assert abs(r["dirty"] - p) < 0.02 * n, (r, p)
        assert r["dirty"] / n == pytest.approx(0.777, abs=0.02)
    # the pause makes the final round exact
    assert torch.equal(dest, cur.view(-1).view(torch.uint8))
    assert torch.equal(shipped, dest)


def test_driver_without_writes_ships_once(wm):
    from paper_2607_10389_amd import Mover, precopy
    cur = wm_inputs.make_cache(wm_inputs.TINY, "cuda")
    nbytes = wm_inputs.TINY.nbytes
    shipped = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dest = torch.zeros_like(shipped)
    m = Mover(nbytes)
    rounds = precopy.run(m, cur, shipped, dest, lambda k, nd: None, stop_chunks=0,
                         max_rounds=5)
    # round 0 ships every chunk, round 1 finds nothing dirty, the final
    # round after the pause ships nothing
    assert [r["dirty"] for r in rounds] == [nbytes // CH, 0, 0]
    assert torch.equal(dest, cur.view(-1).view(torch.uint8))


def test_rounds_while_the_source_keeps_writing(wm):
    """The source is rewritten on another stream while rounds run (chunk
    writes racing the rounds' reads); after the writer stops, one more round
    makes the destination equal to the source, byte for byte."""
    from paper_2607_10389_amd import Mover, precopy
    spec = SPEC
    cur = wm_inputs.make_cache(spec, "cuda")
    nbytes, n = spec.nbytes, spec.nbytes // CH
    shipped = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    dest = torch.zeros_like(shipped)
    m = Mover(nbytes)
    writer = torch.cuda.Stream()
    torch.cuda.synchronize()
    dirty = []
    for k in range(6):
        with torch.cuda.stream(writer):  # enqueued, runs alongside the round
            for b in range(4):
                ids = wm_inputs.chunk_writes(n, 256, seed=7000 + 10 * k + b, device="cuda")
                wm_inputs.rewrite_chunks(cur, spec, ids, seed=8000 + 10 * k + b)
        st, nd = m.precopy_round(cur, shipped, dest)
        assert st == wm.WM_OK
        dirty.append(nd)
    writer.synchronize()  # the pause
    rounds = precopy.run(m, cur, shipped, dest, lambda k, nd: None, stop_chunks=0, max_rounds=3)
    say(f"[precopy] racing rounds: {dirty}, then {[r['dirty'] for r in rounds]}")
    assert torch.equal(dest, cur.view(-1).view(torch.uint8))
    assert torch.equal(shipped, dest)
    assert rounds[-1]["dirty"] == 0
