"""Benchmark: GB/s of KV cache checksummed+encoded and decoded+verified on one
MI355X.

One step = the whole hot path on the production-size cache
([28, 2, 16, 7296, 128] bf16, 1,673,527,296 bytes, synthetic, seeded):
source side wm_encode_step (per-chunk CRC + global CRC + encode of every
chunk, one pass), destination side wm_decode_verify (decode fused with the
CRC check) and wm_commit_or_abort (verdict read back; the full ship's shadow
buffer is then swapped in).  value = state bytes x steps / wall time of the
timed steps.  Inputs are resident in HBM before timing starts.

Also reported: per-side kernel times (HIP events on the launch stream), the
roofline of the dominant side, the compression ratio, the active-generation
step (75% of chunks rewritten: dirty diff + checksum + encode of the dirty
chunks, decode + verify + scatter install), and the CPU oracle on a bounded
sample of the same cache.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X published HBM3E bandwidth


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true",
                    help="skip the CPU oracle baseline")
    ap.add_argument("--no-step", action="store_true",
                    help="skip the active-generation step measurement")
    ap.add_argument("--no-manifest", action="store_true",
                    help="skip the 450-leaf flatten/rehydrate measurement")
    ap.add_argument("--no-fanin", action="store_true",
                    help="skip the eight-session fan-in measurement")
    ap.add_argument("--no-v2", action="store_true",
                    help="skip the format v2 and v3 (Huffman-coded plane) measurements")
    ap.add_argument("--no-receive", action="store_true",
                    help="skip the pipelined receive measurement")
    ap.add_argument("--no-precopy", action="store_true",
                    help="skip the iterative pre-copy measurement")
    ap.add_argument("--no-long", action="store_true",
                    help="skip the 4.3 GB long-context ship and its abort path")
    ap.add_argument("--crc", type=int, default=0, help="0 zlib CRC-32, 1 CRC-32C")
    ap.add_argument("--counter-pass", action="store_true",
                    help="one full-ship encode and decode plus a 1 GiB device copy, "
                         "nothing timed (for rocprofv3 --pmc runs)")
    return ap.parse_args()


KERNELS_SRC = os.path.join(ROOT, "paper_2607_10389_amd", "csrc", "wm_kernels.hip")
TRAFFIC = os.path.join(ROOT, "profiles", "hbm_traffic_production.json")


def kernels_sha256():
    import hashlib
    with open(KERNELS_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter runs
    (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy), or None when the
    kernels changed since they were taken."""
    try:
        with open(TRAFFIC) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernels_sha256") != kernels_sha256() or kernel not in t.get("kernels", {}):
        return None
    k = t["kernels"][kernel]
    return int(k["fetch_bytes"] + k["write_bytes"])


def counter_pass(args):
    """Exactly one launch of each hot kernel on the production cache, a plain
    device-to-device copy of 1 GiB (the calibration for FETCH_SIZE and
    WRITE_SIZE), one flatten and one rehydrate of the 450-leaf manifest,
    then one format v2 encode (CRCs given) and decode."""
    import torch

    import wm_inputs
    from paper_2607_10389_amd import Mover, WM_OK, _wm

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    state = wm_inputs.make_cache(wm_inputs.PRODUCTION, dev)
    m = Mover(state.numel() * 2, args.crc, dev)
    src = torch.randint(0, 255, (1 << 30,), dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    m.encode_step(state, None)
    m.decode()
    ok = m.commit(None, scatter=False) == WM_OK
    dst.copy_(src)
    leaves = wm_inputs.make_manifest(wm_inputs.PRODUCTION, dev, cache=state)
    flat = torch.empty(_wm.flat_bytes(leaves), dtype=torch.uint8, device=dev)
    ws = torch.empty(_wm.manifest_ws_bytes(len(leaves)), dtype=torch.uint8, device=dev)
    _wm.flatten(leaves, flat, ws)
    _wm.rehydrate(flat, leaves, ws)
    del leaves, flat
    m2 = Mover(state.numel() * 2, args.crc, dev, codec=_wm.WM_CODEC_EXPHUF)
    m2.checksum(state)
    m2.encode(state)
    m2.decode()
    ok = ok and m2.commit(None, scatter=False) == WM_OK
    torch.cuda.synchronize()
    print(json.dumps({"counter_pass": "done", "verified": ok, "copy_bytes": src.numel(),
                      "payload_bytes": int(m.payload_bytes.item()),
                      "state_bytes": state.numel() * 2}), flush=True)


# GPU clock cycles of the spin that each timed run waits behind (about 0.45
# ms at the shader clock): long enough for the host to enqueue a whole call,
# Python binding included, before the GPU reaches it.
PREROLL_CYCLES = 1_000_000


def timed_events(torch, fn, n, warmup=3, preroll=True):
    """Median duration (ms) of fn() over n runs, each bracketed by its own
    pair of HIP events on the current stream, after `warmup` untimed runs.

    With `preroll`, each run is queued behind a short spin kernel, so that
    the host has enqueued the start event, every launch of the call and the
    end event before the GPU reaches them: the bracket then holds the call's
    device time (all of its launches and the device's gaps between them)
    and not the host's launch latency, which a caller that keeps the GPU
    busy never sees.  Without it the GPU starts each run idle and waits for
    the host between launches."""
    for _ in range(warmup):
        fn()
    s = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(n):
        if preroll:
            torch.cuda._sleep(PREROLL_CYCLES)
        s.record()
        fn()
        e.record()
        e.synchronize()
        times.append(s.elapsed_time(e))
    times.sort()
    return times[n // 2] if n % 2 else 0.5 * (times[n // 2 - 1] + times[n // 2])


def cpu_threads() -> int:
    """Threads the CPU oracle runs with: every CPU this process may run on
    (its affinity mask), capped by OMP_NUM_THREADS when that is set (the
    share of the host a GPU job is given)."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS", "")
    return min(n, int(cap)) if cap.isdigit() and int(cap) > 0 else n


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(host_state, nbytes_chunk=65536, target_s=12.0):
    """The oracle (as it stands) on the first m chunks of the cache, m sized
    for about target_s seconds of work; round trip = encode (per-chunk CRCs,
    global CRC, records) + decode_verify + commit."""
    import numpy as np

    import oracle
    threads = cpu_threads()

    def run(m):
        sample = host_state[: m * nbytes_chunk]
        t0 = time.perf_counter()
        payload = oracle.encode(0, sample, nbytes_chunk, None, threads)
        v, staging, _ = oracle.decode_verify(0, payload, sample.size,
                                             nbytes_chunk, None, threads)
        live = np.zeros_like(sample)
        rc = oracle.commit(live, nbytes_chunk, staging, payload, v)
        dt = time.perf_counter() - t0
        assert v == 0 and rc == 0 and np.array_equal(live, sample)
        return dt

    m = 64
    dt = run(m)
    n_total = host_state.size // nbytes_chunk
    m = int(min(n_total, max(64, m * target_s / max(dt, 1e-3))))
    dt = run(m)
    gbs = m * nbytes_chunk / dt / 1e9
    cpu = cpu_model()
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"first {m} of {n_total} 64 KiB chunks of the production "
                      f"cache ({m * nbytes_chunk} B); encode + decode_verify + "
                      f"commit, {dt:.1f} s",
            "cpu_model": cpu,
            "threads_rule": "len(os.sched_getaffinity(0)), capped by OMP_NUM_THREADS if set",
            "affinity_cpus": len(os.sched_getaffinity(0))}


def cpu_oracle_detail(host_prev, host_cur, tiny_prev, tiny_cur, host_long, threads):
    """The oracle per operation, in GB/s of state bytes: checksum, diff,
    encode (full ship) and decode + verify.  Each rate is the median of at
    least three timed runs (with their minimum and maximum).  Tiny cache:
    whole, one thread and `threads`.  Production cache: a labelled sample of
    its first chunks with one thread and with `threads` (the whole cache
    takes minutes per operation at one thread).  Long-context cache: a
    labelled sample with `threads` only."""
    import statistics

    import oracle
    CH = 65536

    def rate(fn, nbytes, min_s=0.3, reps_min=3):
        ts = []
        t_all = time.perf_counter()
        while len(ts) < reps_min or time.perf_counter() - t_all < min_s:
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return {"median": round(nbytes / statistics.median(ts) / 1e9, 4),
                "min": round(nbytes / max(ts) / 1e9, 4),
                "max": round(nbytes / min(ts) / 1e9, 4), "runs": len(ts)}

    def ops(prev, cur, T, with_diff=True):
        payload = oracle.encode(0, cur, CH, None, T)
        out = {
            "checksum": rate(lambda: oracle.checksum_chunks(0, cur, CH, T), cur.size),
            "encode": rate(lambda: oracle.encode(0, cur, CH, None, T), cur.size),
            "decode_verify": rate(lambda: oracle.decode_verify(0, payload, cur.size, CH,
                                                               None, T), cur.size),
        }
        if with_diff:
            out["diff"] = rate(lambda: oracle.diff_dirty(cur, prev, CH, T), cur.size)
        return out

    prod_n = 1024  # chunks of the sample: 64 MiB
    sp, sc = host_prev[: prod_n * CH], host_cur[: prod_n * CH]
    long_n = 1024
    sl = host_long[: long_n * CH]
    return {
        "unit": "GB/s of state bytes (median of >= 3 runs; min and max)",
        "threads": threads,
        "cpu_model": cpu_model(),
        "tiny_one_thread": ops(tiny_prev, tiny_cur, 1),
        "tiny_all_threads": ops(tiny_prev, tiny_cur, threads),
        "production_sample": f"first {prod_n} of {host_cur.size // CH} 64 KiB chunks "
                             f"({prod_n * CH} B) of the production cache and of its "
                             "75%-dirty step",
        "production_one_thread": ops(sp, sc, 1),
        "production_all_threads": ops(sp, sc, threads),
        "long_context_sample": f"first {long_n} of 65536 64 KiB chunks "
                               f"({long_n * CH} B) of the long-context cache (Student-t(3), "
                               "10% of chunks uniform random bits)",
        "long_context_all_threads": ops(None, sl, threads, with_diff=False),
    }


def fanin_run(torch, wm_inputs, crc, dev, reps=5):
    """Eight independent sessions ([24,2,8,4096,128] bf16, 402,653,184 B
    each, seeds 100..107), each encoded (full ship) and decoded with
    verification on its own HIP stream, all enqueued together; wall time
    from a synchronised start to the last stream's end."""
    from paper_2607_10389_amd import Mover, WM_OK

    states = [wm_inputs.make_cache(s, dev) for s in wm_inputs.FANIN]
    streams = [torch.cuda.Stream() for _ in states]
    movers = [Mover(s.numel() * 2, crc, dev, stream=st) for s, st in zip(states, streams)]
    # the caches and buffers were made on the current stream, which the
    # sessions' streams do not wait for
    torch.cuda.synchronize()

    # each session's own time: a pair of events on its stream around its
    # encode and decode
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in states]

    def run(timed=False):
        for i, (m, s, st) in enumerate(zip(movers, states, streams)):
            with torch.cuda.stream(st):
                if timed:
                    ev[i][0].record(st)
                m.encode_step(s, None)
                m.decode()
                if timed:
                    ev[i][1].record(st)

    run()
    torch.cuda.synchronize()
    for m, s in zip(movers, states):
        if m.commit(None, scatter=False) != WM_OK or \
                not torch.equal(m.staging[: m.nbytes], s.view(-1).view(torch.uint8)):
            raise RuntimeError("fan-in session did not verify")
    t0 = time.perf_counter()
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / reps
    per_session_ms = [[] for _ in states]
    for _ in range(reps):
        run(timed=True)
        torch.cuda.synchronize()
        for i, (e0, e1) in enumerate(ev):
            per_session_ms[i].append(e0.elapsed_time(e1))
    sess_ms = [sorted(x)[len(x) // 2] for x in per_session_ms]

    def run_serial():  # the same work, one session after another on one stream
        for m, s in zip(movers, states):
            m.stream = None
            m.encode_step(s, None)
            m.decode()

    run_serial()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        run_serial()
    torch.cuda.synchronize()
    serial = (time.perf_counter() - t0) / reps
    # eight streams on disjoint slices of the CUs: each session keeps its own
    from paper_2607_10389_amd import streams as cu_streams
    parts = cu_streams.partition(len(states))
    for m, cs in zip(movers, parts):
        m.stream = cs.stream

    def run_parts(timed=False):
        for i, (m, s) in enumerate(zip(movers, states)):
            if timed:
                ev[i][0].record(m.stream)
            m.encode_step(s, None)
            m.decode()
            if timed:
                ev[i][1].record(m.stream)

    run_parts()
    torch.cuda.synchronize()
    for m, s in zip(movers, states):
        if m.commit(None, scatter=False) != WM_OK or \
                not torch.equal(m.staging[: m.nbytes], s.view(-1).view(torch.uint8)):
            raise RuntimeError("fan-in session on a CU slice did not verify")
    t0 = time.perf_counter()
    for _ in range(reps):
        run_parts()
    torch.cuda.synchronize()
    parted = (time.perf_counter() - t0) / reps
    part_ms = [[] for _ in states]
    for _ in range(reps):
        run_parts(timed=True)
        torch.cuda.synchronize()
        for i, (e0, e1) in enumerate(ev):
            part_ms[i].append(e0.elapsed_time(e1))
    part_sess_ms = [sorted(x)[len(x) // 2] for x in part_ms]
    for cs in parts:
        cs.close()
    each = states[0].numel() * 2
    return {
        "cu_partitioned_ms": round(parted * 1e3, 3),
        "cu_partitioned_kv_GBps": round(8 * each / parted / 1e9, 1),
        "cu_partitioned_per_session_ms": [round(t, 3) for t in part_sess_ms],
        "cu_partitioned_per_session_kv_GBps": [round(each / (t * 1e-3) / 1e9, 1)
                                               for t in part_sess_ms],
        "workload": "8 sessions x [24,2,8,4096,128] bf16 (402,653,184 B each) on 8 streams: "
                    "full checksum + encode + decode + verify",
        "ms": round(wall * 1e3, 3),
        "aggregate_kv_GBps": round(8 * each / wall / 1e9, 1),
        "per_session_ms": [round(t, 3) for t in sess_ms],
        "per_session_kv_GBps": [round(each / (t * 1e-3) / 1e9, 1) for t in sess_ms],
        "per_session_note": "each session's S_i / t_i, t_i between events on its own "
                            "stream around its encode and decode (median of the runs)",
        "one_stream_back_to_back_ms": round(serial * 1e3, 3),
        "one_stream_back_to_back_kv_GBps": round(8 * each / serial / 1e9, 1),
    }


def long_context_run(torch, wm_inputs, crc, dev, one):
    """The long-context cache ([32,2,8,32768,128] bf16, 4,294,967,296 B,
    Student-t(3), 10% of chunks uniform random bits): full ship (encode,
    decode + verify), then the abort path: one payload bit flipped (position
    uniform over the payload's bits, seed 6), decode + verify + scatter
    commit, which must return WM_VERIFY_FAILED with live untouched.  Also
    returns the first 1,024 chunks in host memory for the CPU oracle."""
    import numpy as np

    from paper_2607_10389_amd import Mover, WM_OK, WM_VERIFY_FAILED

    state = wm_inputs.make_cache(wm_inputs.LONG, dev)
    nbytes = state.numel() * 2
    m = Mover(nbytes, crc, dev)
    live = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    m.encode_step(state, None)
    m.decode()
    if m.commit(None, scatter=False) != WM_OK or \
            not torch.equal(m.staging[:nbytes], state.view(-1).view(torch.uint8)):
        raise RuntimeError("long-context ship did not verify")
    pb = int(m.payload_bytes.item())
    src = one("source", lambda: m.encode_step(state, None), nbytes + pb)
    dst = one("destination", lambda: m.decode(), pb + nbytes)
    # modes of the records (byte 0 of each record header), read from the table
    n_rec = nbytes // 65536
    table = m.payload[pb - 16 * n_rec: pb].cpu().numpy().view(np.uint64).reshape(-1, 2)
    offs = torch.from_numpy(table[:, 1].astype(np.int64)).to(dev)
    n_raw = int((m.payload[offs] == 0).sum().item())
    bit = int(np.random.default_rng(6).integers(0, pb * 8))
    m.payload[bit // 8] ^= 1 << (bit % 8)

    def abort():
        m.decode()
        if m.commit(live, scatter=True) != WM_VERIFY_FAILED:
            raise RuntimeError("a flipped payload bit was not rejected")

    t_abort = timed_events(torch, abort, 5, warmup=1)
    verdict = int(m.verdict.item())
    untouched = not bool(live.any())
    m.payload[bit // 8] ^= 1 << (bit % 8)
    if not untouched or verdict == 0:
        raise RuntimeError("the abort path installed something")
    host_sample = state.view(-1).view(torch.uint8)[: 1024 * 65536].cpu().numpy()
    del state, m, live
    torch.cuda.synchronize()
    return {
        "workload": "long-context cache [32,2,8,32768,128] bf16 (4,294,967,296 B), "
                    "Student-t(3), 10% of chunks uniform random 16-bit patterns",
        "payload_bytes": pb, "compression_ratio": round(pb / nbytes, 5),
        "raw_records": n_raw, "records": n_rec,
        "source_wm_encode_step": src,
        "destination_wm_decode_verify": dst,
        "kv_GBps_round_trip": round(nbytes / ((src["ms"] + dst["ms"]) * 1e-3) / 1e9, 1),
        "abort": {"flipped_bit": bit, "verdict": verdict, "live_untouched": untouched,
                  "ms": round(t_abort, 4),
                  "timed": "wm_decode_verify + wm_commit_or_abort (scatter) returning "
                           "WM_VERIFY_FAILED; the commit waits for the stream"},
    }, host_sample


def codec_v2_run(torch, state, nbytes, crc, dev, one, codec=None):
    """Format v2 (per-chunk Huffman codes of the exponents) or v3 (of the
    bf16 high-byte plane) on the production cache: full-ship encode with the
    CRCs computed in the call, decode with verification, and the payload
    ratio (next to format v1's in the same line)."""
    from paper_2607_10389_amd import Mover, WM_CODEC_EXPHUF, WM_OK

    codec = WM_CODEC_EXPHUF if codec is None else codec
    name = "v2" if codec == WM_CODEC_EXPHUF else "v3"
    m = Mover(nbytes, crc, dev, codec=codec)
    m.encode(state, with_crc=False)
    m.decode()
    if m.commit(None, scatter=False) != WM_OK:
        raise RuntimeError(f"format {name} payload did not verify")
    torch.cuda.synchronize()
    if not torch.equal(m.staging[:nbytes], state.view(-1).view(torch.uint8)):
        raise RuntimeError(f"format {name} decode differs from the source")
    pb = int(m.payload_bytes.item())
    return {
        "workload": f"production-size cache, full ship, format {name}",
        "payload_bytes": pb,
        "compression_ratio": round(pb / nbytes, 5),
        "wm_encode": one("enc", lambda: m.encode(state, with_crc=False), nbytes + pb),
        "wm_decode_verify": one("dec", lambda: m.decode(), pb + nbytes),
    }


def receive_runs(torch, m_src, nbytes, crc, dev):
    """The full-ship payload of the production cache arriving in pinned host
    memory: the plain host-to-device copy (the wire), copy then decode on one
    stream (sequential), and wm_receive_verify with record batches of 16, 64
    and 256 MiB (copies on a second stream, each batch decoded as it
    lands).  HIP events on the decode stream bracket each run."""
    from paper_2607_10389_amd import Mover

    pb = int(m_src.payload_bytes.item())
    host = torch.empty(pb, dtype=torch.uint8, pin_memory=True)
    host.copy_(m_src.payload[:pb])
    m = Mover(nbytes, crc, dev)
    cs = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    torch.cuda.synchronize()  # m's buffers are cleared on main, the copies run on cs

    def timed(fn, reps=5):
        """Mean (total ms, ms from the last copy's end to the end of the
        decode) over reps; copies run on cs, the decode on main."""
        fn()
        torch.cuda.synchronize()
        tot = tail = 0.0
        for _ in range(reps):
            s, ec, e = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            s.record(main)
            cs.wait_event(s)
            fn()
            ec.record(cs)
            e.record(main)
            e.synchronize()
            ec.synchronize()
            tot += max(s.elapsed_time(e), s.elapsed_time(ec))
            tail += ec.elapsed_time(e)
        return tot / reps, tail / reps

    def wire():
        with torch.cuda.stream(cs):
            m.payload[:pb].copy_(host, non_blocking=True)

    def sequential():
        wire()
        main.wait_stream(cs)
        m.decode()

    wire_ms, _ = timed(wire)
    seq_ms, seq_tail = timed(sequential)
    torch.cuda.synchronize()
    dec_ms = timed_events(torch, lambda: m.decode(), 10)
    out = {"workload": f"full-ship payload of the production cache ({pb} B) in pinned host memory",
           "wire_ms": round(wire_ms, 3), "wire_GBps": round(pb / wire_ms / 1e6, 2),
           "decode_only_ms": round(dec_ms, 4),
           "sequential": {"ms": round(seq_ms, 3), "exposed_after_last_copy_ms": round(seq_tail, 4)}}
    for mib in (16, 64, 256):
        def piped():
            m.receive(host, pb, mib << 20, cs)
        t, tail = timed(piped)
        if int(m.verdict.item()) != 0 or not torch.equal(m.payload[:pb], m_src.payload[:pb]):
            raise RuntimeError("pipelined receive did not verify")
        out[f"pipelined_{mib}MiB"] = {
            "ms": round(t, 3), "verified_GBps": round(pb / t / 1e6, 2),
            "exposed_after_last_copy_ms": round(tail, 4),
            "one_batch_decode_ms": round(dec_ms * min(1.0, (mib << 20) / pb), 4)}
    return out


def precopy_runs(torch, wm_inputs, spec, state, crc, dev, rho, max_rounds):
    """Iterative pre-copy of the production cache into an empty destination
    while the source writes rho random chunks per chunk shipped (occupancy
    model), until a round ships at most 64 chunks or max_rounds live rounds
    ran; then the final (paused) round.  Each round is one synchronous
    wm_precopy_round, timed with HIP events on its stream."""
    from paper_2607_10389_amd import Mover, _wm
    import math

    nbytes, n = spec.nbytes, spec.nbytes // 65536
    cur = state.clone()
    shipped = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    dest = torch.zeros_like(shipped)
    m = Mover(nbytes, crc, dev)
    rounds, paused, k = [], False, 0
    while True:
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record()
        st, nd = m.precopy_round(cur, shipped, dest)
        e.record()
        e.synchronize()
        if st != _wm.WM_OK:
            raise RuntimeError("pre-copy round failed verification")
        rounds.append({"dirty": nd, "ms": round(s.elapsed_time(e), 4),
                       "payload_bytes": int(m.payload_bytes.item())})
        if paused:
            break
        ids = wm_inputs.chunk_writes(n, int(round(rho * nd)), seed=5000 + k, device=dev)
        wm_inputs.rewrite_chunks(cur, spec, ids, seed=6000 + k)
        k += 1
        paused = nd <= 64 or k >= max_rounds
    torch.cuda.synchronize()
    if not torch.equal(dest, cur.view(-1).view(torch.uint8)):
        raise RuntimeError("pre-copy destination differs from the source")
    # occupancy law for each round after the first, given the previous
    # round's dirty count: w = rho * d writes dirty N (1 - e^(-w/N)) chunks
    pred = [n * (1 - math.exp(-round(rho * r["dirty"]) / n)) for r in rounds[:-1]]
    return {
        "workload": f"production cache into an empty destination, {rho} random chunk "
                    "writes per chunk shipped, pause at <= 64 dirty chunks or "
                    f"{max_rounds} live rounds",
        "rounds": len(rounds),
        "dirty_per_round": [r["dirty"] for r in rounds],
        "occupancy_law_expected_from_round_1": [round(x, 1) for x in pred],
        "ms_per_round": [r["ms"] for r in rounds],
        "total_ms": round(sum(r["ms"] for r in rounds), 4),
        "downtime_ms": rounds[-1]["ms"],
        "final_round_dirty": rounds[-1]["dirty"],
    }


def main():
    args = parse()
    if args.counter_pass:
        return counter_pass(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the "
              "mover's hot path is timed on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import wm_inputs
    from paper_2607_10389_amd import Mover, WM_OK, _wm

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    spec = wm_inputs.PRODUCTION
    state = wm_inputs.make_cache(spec, dev)
    nbytes = spec.nbytes
    m = Mover(nbytes, args.crc, dev)
    torch.cuda.synchronize()

    def source():
        m.encode_step(state, None)

    def destination():
        m.decode()

    def step():
        source()
        destination()
        if m.commit(None, scatter=False) != WM_OK:
            raise RuntimeError("verification failed during the benchmark")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    value = nbytes * args.steps / wall / 1e9

    # decoded shadow must equal the source (checked once, outside timing)
    assert torch.equal(m.staging[:nbytes], state.view(-1).view(torch.uint8))
    payload_bytes = int(m.payload_bytes.item())
    ratio = payload_bytes / nbytes

    src_ms = timed_events(torch, source, 10)
    dst_ms = timed_events(torch, destination, 10)
    # the same calls started on an idle GPU (host launch latency included)
    src_idle_ms = timed_events(torch, source, 10, preroll=False)
    dst_idle_ms = timed_events(torch, destination, 10, preroll=False)
    src_bytes = nbytes + payload_bytes
    dst_bytes = payload_bytes + nbytes
    src_gbs = src_bytes / (src_ms * 1e-3) / 1e9
    dst_gbs = dst_bytes / (dst_ms * 1e-3) / 1e9
    # HIP events bracket one C-ABI call on the stream its kernels run on,
    # queued behind a spin (device time); the call's small set-up and
    # finishing launches are timed with the main one
    dom = ("k_encode", src_ms, src_bytes, src_gbs,
           "wm_encode_step: k_encode_prepare, k_encode, k_combine, k_encode_finish") \
        if src_ms >= dst_ms else \
        ("k_decode", dst_ms, dst_bytes, dst_gbs,
         "wm_decode_verify: k_decode_prepare, k_decode, k_combine (table CRC and verdict)")

    out = {
        "metric": "GB/s of KV cache checksummed+encoded and decoded+verified on 1 MI355X",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16",
        "data": "synthetic",
        "config": {
            "workload": "production-size bf16 KV cache [28,2,16,7296,128] "
                        "(1,673,527,296 B, N(0,1) x LogNormal(0,0.5) channels, "
                        "2% outlier channels x20): full checksum + encode + "
                        "decode + verify",
            "state_bytes": nbytes,
            "chunk_bytes": 65536,
            "crc": "crc32c" if args.crc else "crc32-zlib",
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(dom[3], 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(dom[3] / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(dom[0]),
            "kernel": dom[0],
            "timed_launches": dom[4],
            "algorithmic_bytes_per_launch": dom[2],
            "avg_launch_ms": round(dom[1], 4),
        },
        "sides": {
            "source": {"ms": round(src_ms, 4), "algorithmic_bytes": src_bytes,
                       "GBps": round(src_gbs, 1),
                       "frac_hbm_peak": round(src_gbs / HBM_PEAK_GBS, 4),
                       "kv_GBps": round(nbytes / (src_ms * 1e-3) / 1e9, 1),
                       "ms_from_idle": round(src_idle_ms, 4)},
            "destination": {"ms": round(dst_ms, 4), "algorithmic_bytes": dst_bytes,
                            "GBps": round(dst_gbs, 1),
                            "frac_hbm_peak": round(dst_gbs / HBM_PEAK_GBS, 4),
                            "kv_GBps": round(nbytes / (dst_ms * 1e-3) / 1e9, 1),
                            "ms_from_idle": round(dst_idle_ms, 4)},
        },
        "compression_ratio": round(ratio, 5),
        "payload_bytes": payload_bytes,
        "context": {
            "paper_same_node_relocation_ms": 18.8,
            "paper_same_node_hw": "2x H100, Python path (flatten + cudaMemcpy + CRC + rehydrate), 1.67 GB",
            "paper_verified_wire_Gbps": [92.1, 94.8],
            "paper_wire_hw": "2x CloudLab d6515, 100 Gb RoCE, CPU CRC engine",
            "note": "whole-move numbers on other hardware; context only",
        },
    }

    def one(name, fn, moved):
        t = timed_events(torch, fn, 10)
        return {"ms": round(t, 4), "bytes": moved,
                "GBps": round(moved / (t * 1e-3) / 1e9, 1),
                "frac_hbm_peak": round(moved / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    if not args.no_step:
        prev = state
        cur, ids = wm_inputs.production_step(prev)
        live = prev.clone()
        ms = Mover(nbytes, args.crc, dev)
        torch.cuda.synchronize()

        def a_src():
            ms.encode_step(cur, prev)

        def a_dst():
            ms.decode()
            ms.commit(live, scatter=True)

        a_src()
        a_dst()
        torch.cuda.synchronize()
        assert torch.equal(live, cur)
        n_dirty = int(ms.n_dirty.item())
        assert n_dirty == ids.numel()
        a_src_ms = timed_events(torch, a_src, 10)
        a_dst_ms = timed_events(torch, a_dst, 10)
        pb = int(ms.payload_bytes.item())
        dirty_b = n_dirty * 65536
        out["active_step"] = {
            "workload": "75% of 64 KiB chunks regenerated (Bernoulli, seed 3)",
            "dirty_chunks": n_dirty,
            "source_ms": round(a_src_ms, 4),
            "source_algorithmic_GBps": round((2 * nbytes + pb) / (a_src_ms * 1e-3) / 1e9, 1),
            "destination_ms": round(a_dst_ms, 4),
            "destination_algorithmic_GBps": round((pb + 3 * dirty_b) / (a_dst_ms * 1e-3) / 1e9, 1),
            "kv_GBps_round_trip": round(nbytes / ((a_src_ms + a_dst_ms) * 1e-3) / 1e9, 1),
            "payload_bytes": pb,
        }

        # the same step as separate calls, each against its own bytes
        mu = Mover(nbytes, args.crc, dev)
        mu.checksum(cur)
        mu.diff(cur, prev)
        mu.encode(cur, dirty_only=True)
        torch.cuda.synchronize()
        if not torch.equal(mu.payload[:pb], ms.payload[:pb]):
            raise RuntimeError("separate calls and the fused step disagree")
        mu.decode()

        out["separate_calls"] = {
            "wm_checksum_chunks": one("checksum", lambda: mu.checksum(cur), nbytes),
            "wm_diff_dirty": one("diff", lambda: mu.diff(cur, prev), 2 * nbytes),
            "wm_encode_dirty_list": one("encode", lambda: mu.encode(cur, dirty_only=True),
                                        dirty_b + pb),
            "wm_commit_scatter": one("commit", lambda: mu.commit(live, scatter=True),
                                     2 * dirty_b),
        }
        # what a streaming copy reaches on this device (read S + write S):
        # the library's own copy kernel (a flatten of one leaf, the whole
        # state: 64 KiB windows, 512 threads x 8 x 16 B in flight,
        # non-temporal; the scatter install copies the same way), and
        # torch's copy_
        dst = torch.empty_like(cur).view(-1).view(torch.uint8)
        one_leaf = _wm.LeafTable([cur])
        ws1 = torch.empty(_wm.manifest_ws_bytes(1), dtype=torch.uint8, device=dev)
        out["copy_ceiling"] = one("copy", lambda: _wm.flatten(one_leaf, dst, ws1), 2 * nbytes)
        out["copy_ceiling"]["kernel"] = "k_manifest<gather>, one leaf of the whole state"
        torch.cuda.synchronize()
        if not torch.equal(dst, cur.view(-1).view(torch.uint8)):
            raise RuntimeError("the one-leaf flatten did not copy the state")
        out["copy_ceiling"]["torch_copy_"] = one("copy", lambda: dst.copy_(cur.view(-1).view(torch.uint8)), 2 * nbytes)
        del cur, live, ms, mu, dst

    if not args.no_manifest:
        # the step on either side of the move: gather the session's leaves
        # into the flat buffer, scatter a flat buffer back into the leaves
        leaves = wm_inputs.make_manifest(spec, dev, cache=state)
        total = _wm.flat_bytes(leaves)
        flat = torch.empty(total, dtype=torch.uint8, device=dev)
        ws = torch.empty(_wm.manifest_ws_bytes(len(leaves)), dtype=torch.uint8, device=dev)
        back = [torch.empty_like(x) for x in leaves]
        t_leaves, t_back = _wm.LeafTable(leaves), _wm.LeafTable(back)
        _wm.flatten(t_leaves, flat, ws)
        _wm.rehydrate(flat, t_back, ws)
        torch.cuda.synchronize()
        if not all(torch.equal(x, y) for x, y in zip(back, leaves)):
            raise RuntimeError("rehydrated leaves differ from the flattened ones")
        out["manifest"] = {
            "workload": f"{len(leaves)} leaves (392 bf16 head-group slabs of the "
                        "production cache, 28 fp32 [7296] tensors, 30 scalar flags)",
            "flat_bytes": total,
            "wm_flatten": one("flatten", lambda: _wm.flatten(t_leaves, flat, ws), 2 * total),
            "wm_rehydrate": one("rehydrate", lambda: _wm.rehydrate(flat, t_back, ws),
                                2 * total),
        }
        del leaves, flat, back

    if not args.no_v2:
        out["codec_v2"] = codec_v2_run(torch, state, nbytes, args.crc, dev, one)
        from paper_2607_10389_amd import WM_CODEC_BYTEPLANE
        out["codec_v3"] = codec_v2_run(torch, state, nbytes, args.crc, dev, one,
                                       codec=WM_CODEC_BYTEPLANE)

    host_long = None
    if not args.no_long:
        out["long_context"], host_long = long_context_run(torch, wm_inputs, args.crc, dev, one)

    if not args.no_fanin:
        out["fan_in"] = fanin_run(torch, wm_inputs, args.crc, dev)

    if not args.no_receive:
        out["receive"] = receive_runs(torch, m, nbytes, args.crc, dev)

    if not args.no_precopy:
        out["precopy"] = {r: precopy_runs(torch, wm_inputs, spec, state, args.crc, dev, rho, cap)
                          for r, rho, cap in (("converging", 0.5, 30), ("saturating", 1.93, 6))}

    if not args.no_cpu:
        host = state.view(-1).view(torch.uint8).cpu().numpy()
        out["cpu_baseline"] = cpu_baseline(host)
        out["cpu_baseline"]["paper_context"] = (
            "the paper's 32-thread CPU zlib CRC engine: 52.6 GB/s (CRC only)")
        # the active-generation step's snapshot pair, and the tiny pair
        cur, _ = wm_inputs.production_step(state)
        host_cur = cur.view(-1).view(torch.uint8).cpu().numpy()
        del cur
        tp, tc, _ = wm_inputs.tiny_step("cpu")
        if host_long is None:
            host_long = wm_inputs.make_cache(wm_inputs.LONG, dev).view(-1).view(
                torch.uint8)[: 1024 * 65536].cpu().numpy()
        out["cpu_oracle_detail"] = cpu_oracle_detail(
            host, host_cur, wm_inputs.as_bytes(tp).numpy(), wm_inputs.as_bytes(tc).numpy(),
            host_long, out["cpu_baseline"]["cores"])

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
