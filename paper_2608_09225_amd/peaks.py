"""Python binding of libkvgov_peaks (ctypes): measured-peak microbenchmarks.

Not part of the KVGov path.  ``valu`` and ``gather`` launch the two kernels
declared in include/kvgov_peaks.h on a torch stream and return the work the
launch does (integer ops, or bytes read); the caller times the launch with
events on the same stream.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvgov_peaks.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "kvgov_peaks.h")
THREADS = 256

_vp, _i32, _i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
_SIGNATURES = {
    "kvgov_peak_valu": (ctypes.c_int, [_vp, _i32, _i32, ctypes.POINTER(_i64), _vp]),
    "kvgov_peak_gather": (ctypes.c_int, [_vp, _i64, _vp, _i32, _i32, ctypes.POINTER(_i64),
                                         _vp]),
}
_LIB = None


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _LIB = L
    return _LIB


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def valu(out: torch.Tensor, grid: int, trips: int, stream=None) -> int:
    """Launches the integer-VALU kernel; returns its op count."""
    if not out.is_cuda or out.dtype != torch.int32 or out.numel() < grid * THREADS:
        raise ValueError("out must be an int32 GPU tensor of grid*256 words")
    ops = _i64()
    rc = lib().kvgov_peak_valu(out.data_ptr(), grid, trips, ctypes.byref(ops), _stream(stream))
    if rc:
        raise RuntimeError(f"kvgov_peak_valu failed ({rc})")
    return ops.value


def gather(table: torch.Tensor, out: torch.Tensor, grid: int, trips: int, stream=None) -> int:
    """Launches the 32-byte random-gather kernel over ``table`` (uint8
    [slots, 32], slots a power of two); returns the bytes it reads."""
    if not table.is_cuda or table.dtype != torch.uint8 or table.dim() != 2 or \
            table.shape[1] != 32 or not table.is_contiguous():
        raise ValueError("table must be a contiguous uint8 GPU tensor [slots, 32]")
    if not out.is_cuda or out.dtype != torch.int32 or out.numel() < grid * THREADS:
        raise ValueError("out must be an int32 GPU tensor of grid*256 words")
    nbytes = _i64()
    rc = lib().kvgov_peak_gather(table.data_ptr(), table.shape[0], out.data_ptr(), grid, trips,
                                 ctypes.byref(nbytes), _stream(stream))
    if rc:
        raise RuntimeError(f"kvgov_peak_gather failed ({rc})")
    return nbytes.value
