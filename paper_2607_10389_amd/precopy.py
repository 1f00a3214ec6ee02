"""Iterative pre-copy driver over wm_precopy_round (§6.2 Exhibit 2; App. H).

Each live round ships the chunks of the source that differ from what the
destination holds, while the source keeps writing.  When a round ships at
most `stop_chunks` chunks, or after `max_rounds` live rounds, the source
pauses and one final round makes the destination bit-identical; the final
round is the move's downtime.  Every step runs in libwm's kernels; this
module only sequences the rounds.
"""
from __future__ import annotations

import time

from . import _wm


def run(mover, cur, shipped, dest, write, stop_chunks: int, max_rounds: int):
    """Pre-copy cur into dest.

    write(k, n_dirty) is the source's activity while live round k was
    shipping n_dirty chunks (it writes cur; it is not called after the
    pause).  shipped and dest must hold the same bytes on entry (e.g. both
    zero).  Returns one dict per round: round, dirty, ms (wall time of the
    synchronous round), live (False for the final round).  Raises WmError if
    a round fails verification (dest and shipped then hold the previous
    round's state)."""
    rounds = []
    for k in range(max(max_rounds, 1)):
        t0 = time.perf_counter()
        st, n = mover.precopy_round(cur, shipped, dest)
        ms = (time.perf_counter() - t0) * 1e3
        if st != _wm.WM_OK:
            raise _wm.WmError(st, f"pre-copy round {k}")
        rounds.append({"round": k, "dirty": n, "ms": ms, "live": True})
        write(k, n)
        if n <= stop_chunks:
            break
    t0 = time.perf_counter()
    st, n = mover.precopy_round(cur, shipped, dest)
    ms = (time.perf_counter() - t0) * 1e3
    if st != _wm.WM_OK:
        raise _wm.WmError(st, "pre-copy final round")
    rounds.append({"round": len(rounds), "dirty": n, "ms": ms, "live": False})
    return rounds
