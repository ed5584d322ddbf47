"""ctypes binding of libsplice_calib.so: one plain stream read of device
memory, the kernel whose rate is the measured HBM read ceiling that the
attention library's bandwidth is reported beside.  Argument marshalling only;
the read runs in the library's HIP kernel, and a missing library is an error.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsplice_calib.so")
MAX_BLOCKS = 65536

_lib = None


class CalibError(RuntimeError):
    pass


def load_library(path: str = LIB_PATH):
    """Load libsplice_calib.so (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is None:
        import torch  # noqa: F401  (the HIP runtime torch loads)
        if not os.path.exists(path):
            raise CalibError(f"{path} is missing: run python -m paper_2605_30574_amd.build")
        lib = ctypes.CDLL(path)
        lib.splice_calib_stream_read.restype = ctypes.c_int32
        lib.splice_calib_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                                                 ctypes.c_int32, ctypes.c_void_p]
        _lib = lib
    return _lib


def stream_read(buf, sink, blocks: int, stream=None) -> None:
    """Enqueue one read of every byte of `buf` (a contiguous device tensor of
    16-byte-aligned storage, size a multiple of 16) on `stream` (a
    torch.cuda.Stream, default: the current one); word b of `sink` (an int32
    device tensor of at least `blocks` elements) receives the XOR of part b."""
    import torch
    lib = load_library()
    if not (buf.is_cuda and sink.is_cuda and buf.is_contiguous() and sink.is_contiguous()):
        raise CalibError("stream_read: buf and sink must be contiguous device tensors")
    if sink.dtype != torch.int32 or sink.numel() < blocks:
        raise CalibError("stream_read: sink must be int32 with at least `blocks` elements")
    s = stream if stream is not None else torch.cuda.current_stream(buf.device)
    rc = lib.splice_calib_stream_read(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                      ctypes.c_void_p(sink.data_ptr()), int(blocks),
                                      ctypes.c_void_p(s.cuda_stream))
    if rc != 0:
        raise CalibError(f"splice_calib_stream_read returned {rc}")
