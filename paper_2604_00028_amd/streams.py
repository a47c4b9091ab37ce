"""HIP streams confined to a subset of the compute units.

cu_margin (the paper's sm_margin, Section 3.1) plans a launch for fewer CUs
than the chip has, so that concurrent work keeps the rest.  On MI355X the
reservation itself is a CU mask on the queue: kernels launched on a masked
stream run only on the enabled CUs (hipExtStreamCreateWithCUMask).  Streams
keep the default priority.
"""

from __future__ import annotations

import ctypes
from typing import List, Tuple

import torch

from ._binding import _hip_runtimes_loaded


def _hip() -> ctypes.CDLL:
    runtimes = _hip_runtimes_loaded()
    if len(runtimes) != 1:
        raise RuntimeError(f"expected one HIP runtime loaded by torch, found {runtimes}")
    lib = ctypes.CDLL(runtimes[0])
    lib.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_uint32)]
    lib.hipExtStreamCreateWithCUMask.restype = ctypes.c_int
    lib.hipExtStreamGetCUMask.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint32)]
    lib.hipExtStreamGetCUMask.restype = ctypes.c_int
    lib.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    lib.hipStreamDestroy.restype = ctypes.c_int
    return lib


def split_masks(num_cus: int, reserved_per_32: int) -> Tuple[List[int], List[int]]:
    """Two complementary CU masks (32-bit words): `reserved_per_32` of every
    32 CU bits (the low ones) for concurrent work, the rest for decode.

    reserved_per_32 must be a multiple of 8 in [8, 24]: then every XCD keeps
    CUs in both masks whether the runtime maps mask bits to XCDs in blocks of
    32 or in turn (bit i on XCD i % 8), so no XCD is left without CUs."""
    if reserved_per_32 % 8 or not 8 <= reserved_per_32 <= 24:
        raise ValueError("reserved_per_32 must be 8, 16 or 24")
    if num_cus % 32:
        raise ValueError("num_cus must be a multiple of 32")
    low = (1 << reserved_per_32) - 1
    n = num_cus // 32
    return [low] * n, [(~low) & 0xFFFFFFFF] * n


def cu_mask_stream(words: List[int]) -> Tuple[torch.cuda.ExternalStream, int]:
    """A new stream on the current device whose kernels run only on the CUs
    whose bits are set.  Returns the stream and the number of CUs the runtime
    reports enabled.  Release it with destroy_stream()."""
    lib = _hip()
    arr = (ctypes.c_uint32 * len(words))(*words)
    handle = ctypes.c_void_p()
    rc = lib.hipExtStreamCreateWithCUMask(ctypes.byref(handle), len(words), arr)
    if rc != 0:
        raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
    got = (ctypes.c_uint32 * len(words))()
    rc = lib.hipExtStreamGetCUMask(handle, len(words), got)
    if rc != 0:
        lib.hipStreamDestroy(handle)
        raise RuntimeError(f"hipExtStreamGetCUMask failed ({rc})")
    return torch.cuda.ExternalStream(handle.value), sum(bin(x).count("1") for x in got)


def destroy_stream(stream: torch.cuda.ExternalStream) -> None:
    torch.cuda.synchronize()
    rc = _hip().hipStreamDestroy(ctypes.c_void_p(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"hipStreamDestroy failed ({rc})")
