"""HIP streams restricted to a slice of the GPU's compute units.

A stream made with hipExtStreamCreateWithCUMask runs its kernels on the CUs
of its mask only; libwm sizes its persistent grids to a stream's mask, so
several sessions on such streams each keep their own CUs instead of taking
turns for the whole GPU.  Plumbing only: no work of the mover runs here.
"""
from __future__ import annotations

import ctypes

import torch

_hip = None


def _lib():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                      ctypes.c_uint32,
                                                      ctypes.POINTER(ctypes.c_uint32)]
        _hip.hipExtStreamCreateWithCUMask.restype = ctypes.c_int
        _hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        _hip.hipStreamDestroy.restype = ctypes.c_int
    return _hip


class CuStream:
    """A stream on CUs [first, first + count) of the current device (the
    mask's bit i is CU i).  Use .stream with torch.cuda.stream() or pass it
    to libwm; call close() when no work on it is pending any more."""

    def __init__(self, first: int, count: int):
        n = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
        if count <= 0 or first < 0 or first + count > n:
            raise ValueError(f"CUs [{first}, {first + count}) outside 0..{n}")
        words = (ctypes.c_uint32 * ((n + 31) // 32))()
        for cu in range(first, first + count):
            words[cu // 32] |= 1 << (cu % 32)
        handle = ctypes.c_void_p()
        rc = _lib().hipExtStreamCreateWithCUMask(ctypes.byref(handle), len(words), words)
        if rc != 0:
            raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
        self._handle = handle
        self.stream = torch.cuda.ExternalStream(handle.value)

    def close(self):
        if self._handle is not None:
            self.stream.synchronize()
            _lib().hipStreamDestroy(self._handle)
            self._handle = None


def partition(n_streams: int) -> list[CuStream]:
    """n_streams streams on disjoint, equal slices of the CUs."""
    n = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    per = n // n_streams
    return [CuStream(i * per, per) for i in range(n_streams)]
