"""ctypes binding of libwm (include/wm.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels of libwm.so.  Tensors are torch CUDA (HIP) tensors; the binding
passes their device pointers, sizes and the current stream's handle.  There
is no CPU fallback: if libwm.so is missing or cannot load, importing this
module raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwm.so")

WM_OK = 0
WM_VERIFY_FAILED = 1
WM_ERR_INVALID_ARG = -1
WM_ERR_CAPACITY = -2
WM_ERR_HIP = -3
WM_ERR_WORKSPACE = -4
WM_ERR_UNSUPPORTED = -5

WM_CRC32_ZLIB = 0
WM_CRC32C = 1
WM_CODEC_EXPFOR = 1
WM_CODEC_EXPHUF = 2
WM_CODEC_BYTEPLANE = 3

V_HEADER, V_TABLE, V_RECORD, V_DATA, V_STAGING, V_REVERIFY = 1, 2, 4, 8, 16, 32

WM_COMMIT_NONE = 0
WM_COMMIT_SCATTER = 1

CHUNK = 65536

# every symbol declared in include/wm.h
EXPORTS = (
    "wm_status_str", "wm_init", "wm_workspace_bytes", "wm_payload_bound",
    "wm_checksum_chunks", "wm_diff_dirty", "wm_encode", "wm_encode_step",
    "wm_decode_verify", "wm_commit_or_abort", "wm_flat_bytes",
    "wm_manifest_ws_bytes", "wm_flatten", "wm_rehydrate", "wm_precopy_round",
    "wm_receive_verify", "wm_encode_step_static", "wm_commit_reverify",
)


class WmError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_str(status)} ({status})")
        self.status = status


class Params(ctypes.Structure):
    _fields_ = [("chunk_bytes", ctypes.c_uint32), ("crc_kind", ctypes.c_uint32),
                ("codec", ctypes.c_uint32), ("flags", ctypes.c_uint32)]


class Leaf(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("bytes", ctypes.c_uint64)]


class MoveBuffers(ctypes.Structure):
    _fields_ = [("crc", ctypes.c_void_p), ("global_crc", ctypes.c_void_p),
                ("dirty_idx", ctypes.c_void_p), ("n_dirty", ctypes.c_void_p),
                ("payload", ctypes.c_void_p), ("payload_cap", ctypes.c_uint64),
                ("payload_bytes", ctypes.c_void_p),
                ("staging", ctypes.c_void_p), ("staging_cap", ctypes.c_uint64),
                ("verdict", ctypes.c_void_p), ("rec_status", ctypes.c_void_p),
                ("ws_src", ctypes.c_void_p), ("ws_src_bytes", ctypes.c_uint64),
                ("ws_dst", ctypes.c_void_p), ("ws_dst_bytes", ctypes.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing; build it with "
            "`python -m paper_2607_10389_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
    pp = ctypes.POINTER(Params)
    lp = ctypes.POINTER(Leaf)
    sig = {
        "wm_status_str": ([ctypes.c_int32], ctypes.c_char_p),
        "wm_init": ([ctypes.c_int], ctypes.c_int32),
        "wm_workspace_bytes": ([u64, pp], u64),
        "wm_payload_bound": ([u64, u32, pp], u64),
        "wm_checksum_chunks": ([vp, u64, pp, vp, vp, vp], ctypes.c_int32),
        "wm_diff_dirty": ([vp, vp, u64, pp, vp, vp, vp, u64, vp], ctypes.c_int32),
        "wm_encode": ([vp, u64, pp, vp, vp, vp, vp, u64, vp, vp, u64, vp],
                      ctypes.c_int32),
        "wm_encode_step": ([vp, vp, u64, pp, vp, vp, vp, vp, vp, u64, vp, vp,
                            u64, vp], ctypes.c_int32),
        "wm_encode_step_static": ([vp, vp, u64, pp, vp, vp, vp, vp, vp, u64, vp,
                                   vp], ctypes.c_int32),
        "wm_decode_verify": ([vp, u64, u64, pp, vp, u64, vp, vp, vp, u64, vp],
                             ctypes.c_int32),
        "wm_commit_or_abort": ([vp, u64, pp, vp, vp, vp, u32, vp],
                               ctypes.c_int32),
        "wm_commit_reverify": ([vp, u64, pp, vp, vp, vp, vp, u64, vp], ctypes.c_int32),
        "wm_flat_bytes": ([lp, u32], u64),
        "wm_manifest_ws_bytes": ([u32], u64),
        "wm_flatten": ([lp, u32, vp, u64, vp, u64, vp], ctypes.c_int32),
        "wm_rehydrate": ([vp, u64, lp, u32, vp, u64, vp], ctypes.c_int32),
        "wm_receive_verify": ([vp, u64, vp, u64, u64, pp, vp, u64, vp, vp, vp, u64,
                               u64, vp, vp], ctypes.c_int32),
        "wm_precopy_round": ([vp, vp, vp, u64, pp, ctypes.POINTER(MoveBuffers), u32,
                              ctypes.POINTER(u32), vp], ctypes.c_int32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


def status_str(s: int) -> str:
    return LIB.wm_status_str(s).decode()


def params(crc_kind: int = WM_CRC32_ZLIB, chunk_bytes: int = CHUNK,
           codec: int = WM_CODEC_EXPFOR) -> Params:
    return Params(chunk_bytes, crc_kind, codec, 0)


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libwm takes device tensors")
    return ctypes.c_void_p(t.data_ptr())


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(status: int, where: str) -> int:
    if status < 0:
        raise WmError(status, where)
    return status


def n_chunks(nbytes: int, chunk: int = CHUNK) -> int:
    return (nbytes + chunk - 1) // chunk


def workspace_bytes(nbytes: int, p: Params | None = None) -> int:
    p = p or params()
    return int(LIB.wm_workspace_bytes(nbytes, ctypes.byref(p)))


def payload_bound(nbytes: int, n_records: int, p: Params | None = None) -> int:
    p = p or params()
    return int(LIB.wm_payload_bound(nbytes, n_records, ctypes.byref(p)))


def init(device: int = -1) -> None:
    _check(LIB.wm_init(device), "wm_init")


def checksum_chunks(data, nbytes, p, crc_out, global_crc=None, stream=None):
    return _check(LIB.wm_checksum_chunks(_p(data), nbytes, ctypes.byref(p),
                                         _p(crc_out), _p(global_crc),
                                         _stream(stream)), "wm_checksum_chunks")


def diff_dirty(cur, prev, nbytes, p, dirty_idx, n_dirty, ws, stream=None):
    return _check(LIB.wm_diff_dirty(_p(cur), _p(prev), nbytes, ctypes.byref(p),
                                    _p(dirty_idx), _p(n_dirty), _p(ws),
                                    _nbytes(ws), _stream(stream)),
                  "wm_diff_dirty")


def encode(state, nbytes, p, idx, n_idx, crc, payload, payload_bytes, ws,
           stream=None):
    return _check(LIB.wm_encode(_p(state), nbytes, ctypes.byref(p), _p(idx),
                                _p(n_idx), _p(crc), _p(payload),
                                _nbytes(payload), _p(payload_bytes), _p(ws),
                                _nbytes(ws), _stream(stream)), "wm_encode")


def encode_step(cur, prev, nbytes, p, crc_out, global_crc, dirty_idx, n_dirty,
                payload, payload_bytes, ws, stream=None):
    return _check(LIB.wm_encode_step(_p(cur), _p(prev), nbytes, ctypes.byref(p),
                                     _p(crc_out), _p(global_crc),
                                     _p(dirty_idx), _p(n_dirty), _p(payload),
                                     _nbytes(payload), _p(payload_bytes),
                                     _p(ws), _nbytes(ws), _stream(stream)),
                  "wm_encode_step")


def encode_step_static(cur, prev, nbytes, p, crc_out, global_crc, dirty_idx,
                       n_dirty, payload, payload_bytes, stream=None):
    """wm_encode_step on the device's built-in workspace (allocates
    nothing; calls on one device must not overlap)."""
    return _check(LIB.wm_encode_step_static(
        _p(cur), _p(prev), nbytes, ctypes.byref(p), _p(crc_out), _p(global_crc),
        _p(dirty_idx), _p(n_dirty), _p(payload), _nbytes(payload),
        _p(payload_bytes), _stream(stream)), "wm_encode_step_static")


def decode_verify(payload, payload_cap, nbytes, p, staging, verdict,
                  rec_status, ws, stream=None):
    return _check(LIB.wm_decode_verify(_p(payload), payload_cap, nbytes,
                                       ctypes.byref(p), _p(staging),
                                       _nbytes(staging) if staging is not None
                                       else 0, _p(verdict), _p(rec_status),
                                       _p(ws), _nbytes(ws), _stream(stream)),
                  "wm_decode_verify")


def commit_or_abort(live, nbytes, p, staging, payload, verdict, mode,
                    stream=None) -> int:
    return _check(LIB.wm_commit_or_abort(_p(live), nbytes, ctypes.byref(p),
                                         _p(staging), _p(payload), _p(verdict),
                                         mode, _stream(stream)),
                  "wm_commit_or_abort")


def commit_reverify(live, nbytes, p, staging, payload, verdict, ws, stream=None):
    """Scatter install after re-verifying the staged records and the global
    CRC of the state it would produce; returns WM_OK or WM_VERIFY_FAILED."""
    return _check(LIB.wm_commit_reverify(_p(live), nbytes, ctypes.byref(p), _p(staging),
                                         _p(payload), _p(verdict), _p(ws), _nbytes(ws),
                                         _stream(stream)), "wm_commit_reverify")


class LeafTable:
    """Host table of (device pointer, byte size) for a list of contiguous
    device tensors; build it once to call flatten/rehydrate repeatedly on the
    same leaves."""

    def __init__(self, leaves):
        self.n = len(leaves)
        self.t = (Leaf * max(self.n, 1))()
        for i, x in enumerate(leaves):
            if not x.is_cuda or not x.is_contiguous():
                raise ValueError("manifest leaves are contiguous device tensors")
            self.t[i].ptr = x.data_ptr()
            self.t[i].bytes = _nbytes(x)


def _table(leaves) -> LeafTable:
    return leaves if isinstance(leaves, LeafTable) else LeafTable(leaves)


def flat_bytes(leaves) -> int:
    tab = _table(leaves)
    return int(LIB.wm_flat_bytes(tab.t, tab.n))


def manifest_ws_bytes(n_leaves: int) -> int:
    return int(LIB.wm_manifest_ws_bytes(n_leaves))


def flatten(leaves, flat, ws, stream=None):
    tab = _table(leaves)
    return _check(LIB.wm_flatten(tab.t, tab.n, _p(flat), _nbytes(flat), _p(ws),
                                 _nbytes(ws), _stream(stream)), "wm_flatten")


def rehydrate(flat, leaves, ws, stream=None):
    tab = _table(leaves)
    return _check(LIB.wm_rehydrate(_p(flat), _nbytes(flat), tab.t, tab.n,
                                   _p(ws), _nbytes(ws), _stream(stream)),
                  "wm_rehydrate")


def move_buffers(crc, global_crc, dirty_idx, n_dirty, payload, payload_bytes,
                 staging, verdict, rec_status, ws_src, ws_dst) -> MoveBuffers:
    def a(t):
        return None if t is None else _p(t).value
    return MoveBuffers(a(crc), a(global_crc), a(dirty_idx), a(n_dirty),
                       a(payload), _nbytes(payload), a(payload_bytes),
                       a(staging), _nbytes(staging), a(verdict), a(rec_status),
                       a(ws_src), _nbytes(ws_src), a(ws_dst), _nbytes(ws_dst))


def precopy_round(cur, shipped, dest, nbytes, p, bufs: MoveBuffers,
                  crc_valid: bool = False, stream=None) -> tuple[int, int]:
    """(status, dirty count) of one pre-copy round; waits for the stream."""
    n = ctypes.c_uint32(0)
    st = _check(LIB.wm_precopy_round(_p(cur), _p(shipped), _p(dest), nbytes,
                                     ctypes.byref(p), ctypes.byref(bufs),
                                     1 if crc_valid else 0, ctypes.byref(n),
                                     _stream(stream)),
                "wm_precopy_round")
    return st, int(n.value)


def receive_verify(host_payload, payload_bytes, payload, nbytes, p, staging,
                   verdict, rec_status, ws, batch_bytes, copy_stream, stream=None):
    """host_payload: a CPU uint8 tensor (pinned for DMA copies)."""
    if host_payload.is_cuda or not host_payload.is_contiguous():
        raise ValueError("host_payload is a contiguous host tensor")
    if payload_bytes > _nbytes(host_payload):
        raise ValueError("payload_bytes exceeds the host buffer")
    return _check(LIB.wm_receive_verify(
        ctypes.c_void_p(host_payload.data_ptr()), payload_bytes, _p(payload),
        _nbytes(payload), nbytes, ctypes.byref(p), _p(staging), _nbytes(staging),
        _p(verdict), _p(rec_status), _p(ws), _nbytes(ws), batch_bytes,
        _stream(copy_stream), _stream(stream)), "wm_receive_verify")
