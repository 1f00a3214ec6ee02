"""Buffer-owning helper around the libwm calls.

A ``Mover`` holds the device buffers one session move needs (chunk CRCs,
dirty list, payload, staging, workspace, verdict) for a state of a fixed
size, and sequences the C-ABI calls of the two sides.  It allocates only in
its constructor; every method enqueues libwm work on one stream.
"""
from __future__ import annotations

import torch

from . import _wm


class Mover:
    def __init__(self, nbytes: int, crc_kind: int = _wm.WM_CRC32_ZLIB,
                 device: str | torch.device = "cuda", stream=None,
                 staging_chunks: int | None = None,
                 codec: int = _wm.WM_CODEC_EXPFOR,
                 chunk_bytes: int = _wm.CHUNK):
        self.nbytes = nbytes
        self.p = _wm.params(crc_kind, chunk_bytes=chunk_bytes, codec=codec)
        self.device = torch.device(device)
        self.stream = stream
        n = _wm.n_chunks(nbytes, chunk_bytes)
        self.n_chunks = n
        # records are 64 KiB units: the chunks, or the tiles of larger ones
        n_units = _wm.n_chunks(nbytes)
        self.n_units = n_units
        u32 = dict(dtype=torch.int32, device=self.device)
        self.crc = torch.zeros(max(n, 1), **u32)
        self.global_crc = torch.zeros(1, **u32)
        self.dirty_idx = torch.zeros(max(n, 1), **u32)
        self.n_dirty = torch.zeros(1, **u32)
        self.payload = torch.zeros(_wm.payload_bound(nbytes, n, self.p),
                                   dtype=torch.uint8, device=self.device)
        self.payload_bytes = torch.zeros(1, dtype=torch.int64, device=self.device)
        ws = _wm.workspace_bytes(nbytes, self.p)
        self.ws_src = torch.zeros(ws, dtype=torch.uint8, device=self.device)
        self.ws_dst = torch.zeros(ws, dtype=torch.uint8, device=self.device)
        sc = n_units if staging_chunks is None else staging_chunks
        self.staging = torch.zeros(max(sc, 1) * _wm.CHUNK, dtype=torch.uint8,
                                   device=self.device)
        self.verdict = torch.zeros(1, **u32)
        self.rec_status = torch.zeros(max(n_units, 1), **u32)
        self._bufs = None
        # self.crc holds the CRCs of the last pre-copy round's shipped
        # snapshot (set by a round that returned WM_OK, cleared by any other
        # call that writes self.crc)
        self._crc_of_shipped = None

    # ---- source side
    def checksum(self, state: torch.Tensor):
        self._crc_of_shipped = None
        _wm.checksum_chunks(state, self.nbytes, self.p, self.crc,
                            self.global_crc, self.stream)

    def diff(self, cur: torch.Tensor, prev: torch.Tensor):
        _wm.diff_dirty(cur, prev, self.nbytes, self.p, self.dirty_idx,
                       self.n_dirty, self.ws_src, self.stream)

    def encode(self, state: torch.Tensor, dirty_only: bool = False,
               with_crc: bool = True):
        idx = self.dirty_idx if dirty_only else None
        n_idx = self.n_dirty if dirty_only else None
        crc = self.crc if with_crc else None
        self._crc_of_shipped = None
        _wm.encode(state, self.nbytes, self.p, idx, n_idx, crc, self.payload,
                   self.payload_bytes, self.ws_src, self.stream)

    def encode_step(self, cur: torch.Tensor, prev: torch.Tensor | None):
        self._crc_of_shipped = None
        _wm.encode_step(cur, prev, self.nbytes, self.p, self.crc,
                        self.global_crc, self.dirty_idx, self.n_dirty,
                        self.payload, self.payload_bytes, self.ws_src,
                        self.stream)

    # ---- destination side
    def decode(self, payload: torch.Tensor | None = None,
               payload_cap: int | None = None):
        pl = self.payload if payload is None else payload
        cap = pl.numel() if payload_cap is None else payload_cap
        _wm.decode_verify(pl, cap, self.nbytes, self.p, self.staging,
                          self.verdict, self.rec_status, self.ws_dst,
                          self.stream)

    def commit(self, live: torch.Tensor | None, scatter: bool,
               payload: torch.Tensor | None = None) -> int:
        pl = self.payload if payload is None else payload
        mode = _wm.WM_COMMIT_SCATTER if scatter else _wm.WM_COMMIT_NONE
        return _wm.commit_or_abort(live, self.nbytes, self.p, self.staging, pl,
                                   self.verdict, mode, self.stream)

    def commit_reverify(self, live: torch.Tensor,
                        payload: torch.Tensor | None = None) -> int:
        """Scatter install after re-verifying the staged records and the
        global CRC of the state the install would produce."""
        pl = self.payload if payload is None else payload
        return _wm.commit_reverify(live, self.nbytes, self.p, self.staging, pl,
                                   self.verdict, self.ws_dst, self.stream)

    def receive(self, host_payload: torch.Tensor, payload_bytes: int,
                batch_bytes: int, copy_stream):
        """Copy a payload from host memory into self.payload in batches on
        copy_stream, decoding and verifying each batch on self.stream as it
        lands (the verdict as after decode())."""
        _wm.receive_verify(host_payload, payload_bytes, self.payload, self.nbytes,
                           self.p, self.staging, self.verdict, self.rec_status,
                           self.ws_dst, batch_bytes, copy_stream, self.stream)

    # ---- iterative pre-copy
    def precopy_round(self, cur: torch.Tensor, shipped: torch.Tensor,
                      dest: torch.Tensor) -> tuple[int, int]:
        """One round (diff against shipped, encode, decode, verify, install
        into dest and shipped); returns (status, dirty chunks).  After a
        successful round on the same shipped and dest buffers, the next one
        checksums only its dirty chunks: shipped must then change only
        through these rounds (its chunk CRCs are kept in self.crc)."""
        if self._bufs is None:
            self._bufs = _wm.move_buffers(
                self.crc, self.global_crc, self.dirty_idx, self.n_dirty,
                self.payload, self.payload_bytes, self.staging, self.verdict,
                self.rec_status, self.ws_src, self.ws_dst)
        valid = self._crc_of_shipped is not None and \
            self._crc_of_shipped == (shipped.data_ptr(), dest.data_ptr())
        self._crc_of_shipped = None
        st, n = _wm.precopy_round(cur, shipped, dest, self.nbytes, self.p,
                                  self._bufs, valid, self.stream)
        if st == _wm.WM_OK:
            self._crc_of_shipped = (shipped.data_ptr(), dest.data_ptr())
        return st, n

    # ---- host views (synchronising)
    def payload_host(self):
        n = int(self.payload_bytes.item())
        return self.payload[:n].cpu().numpy()

    def crc_host(self):
        return self.crc[: self.n_chunks].cpu().numpy().view("uint32")

    def dirty_host(self):
        m = int(self.n_dirty.item())
        return self.dirty_idx[:m].cpu().numpy().view("uint32")
