"""ctypes binding of libsplash_calib (include/splash_calib.h): achievable-peak
measurements and a clean cache flush for the benchmark.  Argument
marshalling only."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsplash_calib.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_37626_amd.build`")
        import torch  # noqa: F401  (torch's HIP runtime first)
        h = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        h.splash_calib_stream_read.argtypes = [vp, sz, vp, i32, vp]
        h.splash_calib_stream_read.restype = ctypes.c_int
        h.splash_calib_mfma_ops_bytes.argtypes = [i32]
        h.splash_calib_mfma_ops_bytes.restype = sz
        h.splash_calib_mfma_loop.argtypes = [vp, i32, vp, i32, vp]
        h.splash_calib_mfma_loop.restype = ctypes.c_int
        h.splash_calib_mfma_flops.argtypes = [i32, i32]
        h.splash_calib_mfma_flops.restype = ctypes.c_double
        _lib = h
    return _lib


def _check(st: int, what: str) -> None:
    if st != 0:
        raise RuntimeError(f"{what} failed with status {st}")


def stream_read(buf, sink, blocks: int, stream) -> None:
    _check(lib().splash_calib_stream_read(buf.data_ptr(), buf.numel() * buf.element_size(), sink.data_ptr(),
                                          blocks, stream.cuda_stream), "stream_read")


def mfma_ops_bytes(blocks: int) -> int:
    return int(lib().splash_calib_mfma_ops_bytes(blocks))


def mfma_loop(ops, iters: int, sink, blocks: int, stream) -> None:
    _check(lib().splash_calib_mfma_loop(ops.data_ptr(), iters, sink.data_ptr(), blocks, stream.cuda_stream),
           "mfma_loop")


def mfma_flops(blocks: int, iters: int) -> float:
    return float(lib().splash_calib_mfma_flops(blocks, iters))
