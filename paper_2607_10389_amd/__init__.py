"""Exact-state mover hot path for MI355X (gfx950).

Device-side processing of a multi-gigabyte bf16 attention (KV) cache on both
ends of a session move (arXiv 2607.10389, WorldMove): per-chunk CRC, dirty
diff against the last shipped snapshot and lossless encoding on the source;
decode fused with re-checksumming and an all-or-nothing install on the
destination.  The work runs in the HIP kernels of ``libwm.so``; this package
is its Python binding (``_wm``) plus a small buffer-owning helper
(``mover.Mover``).
"""
from . import _wm
from ._wm import (  # noqa: F401
    CHUNK, WM_CODEC_BYTEPLANE, WM_CODEC_EXPFOR, WM_CODEC_EXPHUF, WM_CRC32C, WM_CRC32_ZLIB, WM_COMMIT_NONE,
    WM_COMMIT_SCATTER,
    WM_OK, WM_VERIFY_FAILED, WmError, checksum_chunks, commit_or_abort,
    decode_verify, diff_dirty, encode, encode_step, flat_bytes, flatten,
    manifest_ws_bytes, params, payload_bound, rehydrate, workspace_bytes,
)
from .mover import Mover  # noqa: F401
from . import precopy  # noqa: F401
