"""Achievable-peak probes of MI355X (``libbasp_peak.so``), for the benchmark.

``mfma_bf16_tflops`` times back-to-back bf16 MFMAs on register operands over
the whole chip; ``copy_gbps`` times a streaming device copy of at least 1 GiB.
Both are measurement tools only: the attention share never calls them.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(os.path.dirname(_HERE), "libbasp_peak.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built")
        L = ctypes.CDLL(LIB_PATH)
        L.basp_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                          ctypes.c_void_p]
        L.basp_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
        L.basp_peak_mfma_bf16.restype = ctypes.c_int
        L.basp_peak_copy.restype = ctypes.c_int
        _lib = L
    return _lib


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _time(fn, reps):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ts.sort()
    return ts[len(ts) // 2]


def mfma_bf16_tflops(iters: int = 20000, reps: int = 5) -> float:
    """Median rate of v_mfma_f32_32x32x16_bf16 issued back to back, two waves
    per SIMD on every CU (one 512-thread workgroup per CU)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(cus * 512, dtype=torch.float32, device="cuda")
    call = lambda: lib().basp_peak_mfma_bf16(cus, iters, ctypes.c_void_p(out.data_ptr()),
                                             _stream())
    assert call() == 0
    ms = _time(call, reps)
    flops = cus * 8 * iters * 8 * 32 * 32 * 16 * 2.0
    return flops / (ms * 1e-3) / 1e12


# Launch shapes tried by copy_gbps: (workgroups, vectors in flight per thread).
COPY_SHAPES = ((8192, 4), (16384, 4), (32768, 4), (32768, 8), (8192, 8))


def copy_gbps(nbytes: int = 1 << 30, reps: int = 5, shapes=COPY_SHAPES) -> float:
    """Best over launch shapes of the median rate (bytes read + written) of a
    streaming copy of nbytes."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    best = 0.0
    for blocks, unroll in shapes:
        dst.zero_()
        call = lambda: lib().basp_peak_copy(ctypes.c_void_p(src.data_ptr()),
                                            ctypes.c_void_p(dst.data_ptr()), nbytes, blocks,
                                            unroll, _stream())
        assert call() == 0
        ms = _time(call, reps)
        if not bool(torch.equal(src, dst)):
            raise RuntimeError("peak copy produced a wrong result")
        best = max(best, 2.0 * nbytes / (ms * 1e-3) / 1e9)
    del src, dst
    return best
