"""The C ABI without a GPU: libwm.so loads, exports every function that
include/wm.h declares, and its host-side argument checks return the documented
status codes before any device work.  Addresses passed here are never
dereferenced (every call fails validation first)."""
import ctypes
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_10389_amd", "libwm.so")
HEADER = os.path.join(ROOT, "include", "wm.h")

OK, VERIFY_FAILED, INVALID, CAPACITY, HIP, WORKSPACE, UNSUPPORTED = 0, 1, -1, -2, -3, -4, -5
CH = 65536
ALIGNED = 0x7f0000001000  # a well-formed 16-byte aligned address, never touched


class Params(ctypes.Structure):
    _fields_ = [("chunk_bytes", ctypes.c_uint32), ("crc_kind", ctypes.c_uint32),
                ("codec", ctypes.c_uint32), ("flags", ctypes.c_uint32)]


class Leaf(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("bytes", ctypes.c_uint64)]


class MoveBuffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64 if n.endswith(("_cap", "_bytes")) and n != "payload_bytes"
                 else ctypes.c_void_p)
                for n in ("crc", "global_crc", "dirty_idx", "n_dirty", "payload", "payload_cap",
                          "payload_bytes", "staging", "staging_cap", "verdict", "rec_status",
                          "ws_src", "ws_src_bytes", "ws_dst", "ws_dst_bytes")]


def leaves(*pairs):
    t = (Leaf * max(len(pairs), 1))()
    for i, (p, b) in enumerate(pairs):
        t[i].ptr, t[i].bytes = p, b
    return t


def declared():
    text = open(HEADER).read()
    return re.findall(r"^\s*(?:const\s+char\s*\*|wm_status|uint64_t)\s*(wm_\w+)\s*\(",
                      text, flags=re.M)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.skip("libwm.so is not built")
    L = ctypes.CDLL(LIB)
    vp, u64, u32, pp = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.POINTER(Params)
    L.wm_status_str.restype = ctypes.c_char_p
    L.wm_status_str.argtypes = [ctypes.c_int32]
    L.wm_workspace_bytes.restype = u64
    L.wm_workspace_bytes.argtypes = [u64, pp]
    L.wm_payload_bound.restype = u64
    L.wm_payload_bound.argtypes = [u64, u32, pp]
    L.wm_checksum_chunks.argtypes = [vp, u64, pp, vp, vp, vp]
    L.wm_diff_dirty.argtypes = [vp, vp, u64, pp, vp, vp, vp, u64, vp]
    L.wm_encode.argtypes = [vp, u64, pp, vp, vp, vp, vp, u64, vp, vp, u64, vp]
    L.wm_encode_step.argtypes = [vp, vp, u64, pp, vp, vp, vp, vp, vp, u64, vp, vp, u64, vp]
    L.wm_encode_step_static.argtypes = [vp, vp, u64, pp, vp, vp, vp, vp, vp, u64, vp, vp]
    L.wm_decode_verify.argtypes = [vp, u64, u64, pp, vp, u64, vp, vp, vp, u64, vp]
    L.wm_commit_or_abort.argtypes = [vp, u64, pp, vp, vp, vp, u32, vp]
    L.wm_commit_reverify.argtypes = [vp, u64, pp, vp, vp, vp, vp, u64, vp]
    lp = ctypes.POINTER(Leaf)
    L.wm_flat_bytes.restype = u64
    L.wm_flat_bytes.argtypes = [lp, u32]
    L.wm_manifest_ws_bytes.restype = u64
    L.wm_manifest_ws_bytes.argtypes = [u32]
    L.wm_flatten.argtypes = [lp, u32, vp, u64, vp, u64, vp]
    L.wm_rehydrate.argtypes = [vp, u64, lp, u32, vp, u64, vp]
    L.wm_receive_verify.argtypes = [vp, u64, vp, u64, u64, pp, vp, u64, vp, vp, vp, u64, u64,
                                    vp, vp]
    L.wm_precopy_round.argtypes = [vp, vp, vp, u64, pp, ctypes.POINTER(MoveBuffers), u32,
                                   ctypes.POINTER(u32), vp]
    for name in declared():
        if name not in ("wm_status_str", "wm_workspace_bytes", "wm_payload_bound",
                        "wm_flat_bytes", "wm_manifest_ws_bytes"):
            getattr(L, name).restype = ctypes.c_int32
    return L


def P(chunk=CH, kind=0, codec=1, flags=0):
    return ctypes.byref(Params(chunk, kind, codec, flags))


def test_header_declares_the_boundary():
    names = declared()
    for must in ("wm_checksum_chunks", "wm_diff_dirty", "wm_encode", "wm_decode_verify",
                 "wm_commit_or_abort", "wm_flatten", "wm_rehydrate"):
        assert must in names
    assert len(names) == len(set(names)) == 18


def test_every_declared_symbol_is_exported(lib):
    for name in declared():
        assert hasattr(lib, name), name


def test_binding_lists_the_same_symbols():
    # the binding's export list is plain text: compare without importing torch
    src = open(os.path.join(ROOT, "paper_2607_10389_amd", "_wm.py")).read()
    block = src[src.index("EXPORTS = ("):src.index(")", src.index("EXPORTS = ("))]
    listed = re.findall(r'"(wm_\w+)"', block)
    assert sorted(listed) == sorted(declared())


def test_status_strings(lib):
    for code, name in ((OK, b"WM_OK"), (VERIFY_FAILED, b"WM_VERIFY_FAILED"),
                       (INVALID, b"WM_ERR_INVALID_ARG"), (CAPACITY, b"WM_ERR_CAPACITY"),
                       (HIP, b"WM_ERR_HIP"), (WORKSPACE, b"WM_ERR_WORKSPACE"),
                       (UNSUPPORTED, b"WM_ERR_UNSUPPORTED")):
        assert lib.wm_status_str(code) == name


@pytest.mark.parametrize("nbytes", [0, 2, CH, CH + 2, 1673527296, 4294967296])
def test_payload_bound_matches_the_oracle(lib, nbytes):
    n = -(-nbytes // CH)
    assert lib.wm_payload_bound(nbytes, n, P()) == oracle.payload_bound(nbytes, CH, n)
    # the workspace holds at least the look-back status, table and CRC arrays
    assert lib.wm_workspace_bytes(nbytes, P()) >= 256 + 32 * max(n, 1)


def test_bad_params_are_rejected_before_device_work(lib):
    a = ALIGNED
    assert lib.wm_payload_bound(CH, 1, P(chunk=3000)) == 0   # not a power of two
    assert lib.wm_workspace_bytes(CH, P(kind=2)) == 0        # unknown CRC
    # a valid power-of-two chunk size other than 64 KiB is not implemented
    assert lib.wm_checksum_chunks(a, CH, P(chunk=4096), a, None, None) == UNSUPPORTED
    assert lib.wm_checksum_chunks(a, CH, P(codec=7), a, None, None) == INVALID
    assert lib.wm_checksum_chunks(a + 4, CH, P(), a, None, None) == INVALID  # misaligned
    assert lib.wm_checksum_chunks(None, CH, P(), a, None, None) == INVALID


def test_encode_argument_checks(lib):
    a, big = ALIGNED, 1 << 40
    ws = lib.wm_workspace_bytes(4 * CH, P())
    bound = lib.wm_payload_bound(4 * CH, 4, P())
    enc = lib.wm_encode
    assert enc(a, 4 * CH + 1, P(), None, None, None, a, bound, a, a, ws, None) == INVALID  # odd
    assert enc(a, 4 * CH, P(), a, None, a, a, bound, a, a, ws, None) == INVALID  # idx w/o n_idx
    # a list without CRCs is valid (the call checksums every chunk); its
    # other arguments are checked as usual
    assert enc(a, 4 * CH, P(), a, a, None, a, bound, a, a, ws - 1, None) == WORKSPACE
    assert enc(a, 4 * CH, P(), None, None, None, a, bound - 1, a, a, ws, None) == CAPACITY
    assert enc(a, 4 * CH, P(), None, None, None, a, bound, a, a, ws - 1, None) == WORKSPACE
    assert enc(a, 4 * CH, P(), None, None, None, a + 8, big, a, a, ws, None) == INVALID
    step = lib.wm_encode_step
    assert step(a, a + 2, 4 * CH, P(), None, None, None, None, a, bound, a, a, ws,
                None) == INVALID
    assert step(a, None, 4 * CH, P(), None, None, None, None, a, bound - 16, a, a, ws,
                None) == CAPACITY


def test_decode_and_commit_argument_checks(lib):
    a = ALIGNED
    ws = lib.wm_workspace_bytes(4 * CH, P())
    dec = lib.wm_decode_verify
    assert dec(a, 1 << 20, 4 * CH, P(), a, 4 * CH, None, None, a, ws, None) == INVALID
    assert dec(a, 1 << 20, 4 * CH, P(), a, 4 * CH, a, None, a, ws - 256, None) == WORKSPACE
    assert dec(a, 1 << 20, 4 * CH + 1, P(), a, 4 * CH, a, None, a, ws, None) == INVALID
    com = lib.wm_commit_or_abort
    assert com(a, 4 * CH, P(), a, a, None, 1, None) == INVALID   # no verdict
    assert com(a, 4 * CH, P(), a, a, a, 2, None) == INVALID      # unknown mode
    assert com(a + 1, 4 * CH, P(), a, a, a, 1, None) == INVALID  # misaligned live


def test_flat_bytes_matches_the_oracle(lib):
    import wm_inputs
    sizes = wm_inputs.ragged_sizes(100, seed=9)
    t = leaves(*[(ALIGNED, s) for s in sizes])
    assert lib.wm_flat_bytes(t, len(sizes)) == oracle.flat_layout(sizes)[1]
    assert lib.wm_flat_bytes(None, 3) == 0
    assert lib.wm_flat_bytes(None, 0) == 0
    assert lib.wm_flat_bytes(leaves((ALIGNED, 1 << 63), (ALIGNED, 1 << 63)), 2) == 0
    assert lib.wm_manifest_ws_bytes(450) == 32 * 450


def test_manifest_argument_checks(lib):
    a = ALIGNED
    t = leaves((a, 100), (a + 4096, 17))
    flat_b, ws_b = 144, 64  # 112 + 32 flat bytes, 2 x 32 table bytes
    for fn, call in (("flatten", lambda t, n, f, cap, w, wb:
                      lib.wm_flatten(t, n, f, cap, w, wb, None)),
                     ("rehydrate", lambda t, n, f, cap, w, wb:
                      lib.wm_rehydrate(f, cap, t, n, w, wb, None))):
        assert call(None, 2, a, flat_b, a, ws_b) == INVALID, fn
        assert call(leaves((a + 8, 100)), 1, a, flat_b, a, ws_b) == INVALID, fn
        assert call(leaves((None, 100)), 1, a, flat_b, a, ws_b) == INVALID, fn
        assert call(t, 2, a + 4, flat_b, a, ws_b) == INVALID, fn
        assert call(t, 2, None, flat_b, a, ws_b) == INVALID, fn
        assert call(t, 2, a, flat_b - 16, a, ws_b) == CAPACITY, fn
        assert call(t, 2, a, flat_b, a, ws_b - 1) == WORKSPACE, fn
        assert call(t, 2, a, flat_b, None, ws_b) == WORKSPACE, fn
        assert call(t, 2, a, flat_b, a + 2, ws_b) == WORKSPACE, fn
        big = leaves((a, (1 << 64) - 8), (a, 64))
        assert call(big, 2, a, 1 << 62, a, ws_b) == INVALID, fn
        # nothing to copy: no device work, so this returns without a GPU
        assert call(None, 0, None, 0, None, 0) == OK, fn
        assert call(leaves((None, 0), (a + 3, 0)), 2, None, 0, a, ws_b) == OK, fn


def test_precopy_round_argument_checks(lib):
    a = ALIGNED
    nb = 4 * CH
    ws = lib.wm_workspace_bytes(nb, P())
    bound = lib.wm_payload_bound(nb, 4, P())

    def bufs(**kw):
        d = dict(crc=a, global_crc=None, dirty_idx=a, n_dirty=a, payload=a + 0x100000,
                 payload_cap=bound, payload_bytes=a, staging=a + 0x200000, staging_cap=nb,
                 verdict=a, rec_status=None, ws_src=a + 0x300000, ws_src_bytes=ws,
                 ws_dst=a + 0x400000, ws_dst_bytes=ws)
        d.update(kw)
        return ctypes.byref(MoveBuffers(**d))

    n = ctypes.c_uint32(0)
    cur, shp, dst = a + 0x500000, a + 0x600000, a + 0x700000
    rnd = lib.wm_precopy_round
    assert rnd(cur, shp, dst, nb, P(), None, 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(), bufs(), 0, None, None) == INVALID
    assert rnd(cur, shp, shp, nb, P(), bufs(), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, cur, dst, nb, P(), bufs(), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp + 8, dst, nb, P(), bufs(), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, None, nb, P(), bufs(), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(), bufs(verdict=None), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(), bufs(n_dirty=None), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(), bufs(staging_cap=nb - CH), 0, ctypes.byref(n),
               None) == CAPACITY
    assert rnd(cur, shp, dst, nb, P(), bufs(ws_dst_bytes=ws - 1), 0, ctypes.byref(n),
               None) == WORKSPACE
    assert rnd(cur, shp, dst, nb, P(), bufs(ws_dst=a + 0x300000), 0, ctypes.byref(n),
               None) == WORKSPACE
    assert rnd(cur, shp, dst, nb, P(), bufs(payload_cap=bound - 1), 0, ctypes.byref(n),
               None) == CAPACITY
    assert rnd(cur, shp, dst, nb + 1, P(), bufs(), 0, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(chunk=4096), bufs(), 0, ctypes.byref(n), None) == UNSUPPORTED
    assert rnd(cur, shp, dst, nb, P(), bufs(), 2, ctypes.byref(n), None) == INVALID
    assert rnd(cur, shp, dst, nb, P(), bufs(ws_src_bytes=ws - 1), 1, ctypes.byref(n),
               None) == WORKSPACE


def test_receive_verify_argument_checks(lib):
    a = ALIGNED
    nb = 4 * CH
    ws = lib.wm_workspace_bytes(nb, P())
    host = ctypes.create_string_buffer(4096)
    h = ctypes.addressof(host)
    rv = lib.wm_receive_verify
    # (host, bytes, payload, cap, nbytes, p, staging, staging_cap, verdict, rec_status,
    #  ws, ws_bytes, batch, copy_stream, stream)
    assert rv(h, 4096, a, 4095, nb, P(), a, nb, a, None, a, ws, 0, None, None) == CAPACITY
    assert rv(None, 4096, a, 4096, nb, P(), a, nb, a, None, a, ws, 0, None, None) == INVALID
    assert rv(h, 4096, a + 4, 4096, nb, P(), a, nb, a, None, a, ws, 0, None, None) == INVALID
    assert rv(h, 4096, a, 4096, nb, P(), a, nb, None, None, a, ws, 0, None, None) == INVALID
    assert rv(h, 4096, a, 4096, nb + 1, P(), a, nb, a, None, a, ws, 0, None, None) == INVALID
    assert rv(h, 4096, a, 4096, nb, P(), a + 8, nb, a, None, a, ws, 0, None, None) == INVALID
    assert rv(h, 4096, a, 4096, nb, P(), a, nb, a, None, a, ws - 1, 0, None, None) == WORKSPACE
    assert rv(h, 4096, a, 4096, nb, P(codec=4), a, nb, a, None, a, ws, 0, None, None) == INVALID


def test_format_v2_calls(lib):
    a = ALIGNED
    nb = 4 * CH
    ws1 = lib.wm_workspace_bytes(nb, P())
    ws2 = lib.wm_workspace_bytes(nb, P(codec=2))
    assert ws2 >= ws1 + 4 * 4 + 16  # a dirty list and its length for the fused step
    assert lib.wm_payload_bound(nb, 4, P(codec=2)) == lib.wm_payload_bound(nb, 4, P())
    assert lib.wm_workspace_bytes(nb, P(codec=4)) == 0
    # format v3 (the byte-plane split) shares format v2's kernels and layout
    assert lib.wm_workspace_bytes(nb, P(codec=3)) == ws2
    assert lib.wm_payload_bound(nb, 4, P(codec=3)) == lib.wm_payload_bound(nb, 4, P())
    bound = lib.wm_payload_bound(nb, 4, P())
    enc = lib.wm_encode
    # the plans need the larger workspace
    assert enc(a, nb, P(codec=2), None, None, None, a, bound, a, a, ws1, None) == WORKSPACE
    # the fused step and pre-copy take format v2 too: a v1-sized workspace
    # is too small for them (checked before any device work)
    assert lib.wm_encode_step(a, None, nb, P(codec=2), None, None, None, None, a, bound, a, a,
                              ws1, None) == WORKSPACE
    n = ctypes.c_uint32(0)
    assert lib.wm_precopy_round(a, a + 0x100000, a + 0x200000, nb, P(codec=2), None, 0,
                                ctypes.byref(n), None) == INVALID  # no buffers
    # only the allocation-free step is format v1 only
    assert lib.wm_encode_step_static(a, None, nb, P(codec=2), None, None, None, None, a, bound,
                                     a, None) == UNSUPPORTED


def test_static_step_refuses_a_state_beyond_its_workspace(lib):
    """wm_encode_step_static's built-in workspace holds 65,536 chunks; a
    larger state is refused on the host before any device work."""
    a = ALIGNED
    nbytes = 65537 * CH
    bound = lib.wm_payload_bound(nbytes, 65537, P())
    fn = lib.wm_encode_step_static
    assert fn(a, None, nbytes, P(), None, None, None, None, a, bound, a, None) == WORKSPACE
    # the usual argument checks come first
    assert fn(a, None, nbytes + 1, P(), None, None, None, None, a, bound, a, None) == INVALID
    assert fn(a, None, nbytes, P(), None, None, None, None, a, bound - 1, a, None) == CAPACITY


def test_reverify_argument_checks(lib):
    a = ALIGNED
    ws = lib.wm_workspace_bytes(4 * CH, P())
    rv = lib.wm_commit_reverify
    assert rv(a, 4 * CH, P(), a, a, None, a, ws, None) == INVALID        # no verdict
    assert rv(a + 8, 4 * CH, P(), a, a, a, a, ws, None) == INVALID       # misaligned live
    assert rv(a, 4 * CH, P(), a, a + 4, a, a, ws, None) == INVALID       # misaligned payload
    assert rv(a, 4 * CH, P(), a, a, a, a, ws - 1, None) == WORKSPACE
    assert rv(a, 4 * CH, P(chunk=3000), a, a, a, a, ws, None) == INVALID
