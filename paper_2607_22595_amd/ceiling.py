"""Binding of libxmix_ceiling.so: the device's measured ceilings.

A benchmark aid beside the hook-step library (include/xmix_ceiling.h): a
stream of nontemporal HBM reads and a stream of register-only bf16 MFMAs,
timed by the caller with events.  Nothing in the hook step calls it.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libxmix_ceiling.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP libraries first")
_lib = ctypes.CDLL(LIB_PATH)
_lib.xmix_ceiling_read.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                                   ctypes.c_void_p]
_lib.xmix_ceiling_read.restype = ctypes.c_int
_lib.xmix_ceiling_mfma.argtypes = [ctypes.c_int32, ctypes.c_void_p,
                                   ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
_lib.xmix_ceiling_mfma.restype = ctypes.c_int
EXPORTED = ("xmix_ceiling_read", "xmix_ceiling_mfma")


def _stream(stream) -> int:
    return torch.cuda.current_stream().cuda_stream if stream is None else int(stream)


def read(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> int:
    """Reads all of `buf` (a contiguous device tensor) once; returns its bytes."""
    if not (buf.is_cuda and buf.is_contiguous() and sink.is_cuda and sink.dtype == torch.int32):
        raise ValueError("read: contiguous device buffer and an int32 device sink")
    nbytes = buf.numel() * buf.element_size()
    st = _lib.xmix_ceiling_read(buf.data_ptr(), nbytes, sink.data_ptr(), _stream(stream))
    if st != 0:
        raise RuntimeError(f"xmix_ceiling_read failed (status {st})")
    return nbytes


def mfma(iters: int, sink: torch.Tensor, stream=None) -> float:
    """Runs the MFMA stream; returns the launch's flop count."""
    if not (sink.is_cuda and sink.dtype == torch.float32):
        raise ValueError("mfma: a float32 device sink")
    flops = ctypes.c_double(0.0)
    st = _lib.xmix_ceiling_mfma(iters, sink.data_ptr(), ctypes.byref(flops), _stream(stream))
    if st != 0:
        raise RuntimeError(f"xmix_ceiling_mfma failed (status {st})")
    return flops.value
