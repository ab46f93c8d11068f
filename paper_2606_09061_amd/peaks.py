"""ctypes binding of libcppeaks.so (include/cp_peaks.h): the practical-peak
microbenchmarks.  Argument marshalling only; the kernels run on the GPU."""

from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcppeaks.so")
_lib = None


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                           "(python -m paper_2606_09061_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.cpk_device_info.argtypes = [I32, P, P, P, P]
    lib.cpk_mfma_loop.argtypes = [P, I64, P, I32, I32, I32, I32, P]
    lib.cpk_read_stream.argtypes = [P, I64, P, I32, P]
    for f in (lib.cpk_device_info, lib.cpk_mfma_loop, lib.cpk_read_stream):
        f.restype = ctypes.c_int
    _lib = lib
    return lib


def exported_symbols():
    return ["cpk_device_info", "cpk_mfma_loop", "cpk_read_stream"]


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what} failed ({rc})")


def device_info(device=0) -> dict:
    v = [ctypes.c_int32() for _ in range(4)]
    _check(load().cpk_device_info(device, *[ctypes.byref(x) for x in v]), "cpk_device_info")
    return {"compute_units": v[0].value, "clock_khz": v[1].value, "mem_clock_khz": v[2].value,
            "mem_bus_bits": v[3].value}


def mfma_loop(operands, out, blocks, threads, iters, random_operands, stream):
    """operands: uint8/bf16 device tensor (16-byte elements); out: float32 [blocks*threads]."""
    n16 = operands.numel() * operands.element_size() // 16
    if out.numel() < blocks * threads:
        raise ValueError("out holds fewer than blocks * threads floats")
    _check(load().cpk_mfma_loop(operands.data_ptr(), n16, out.data_ptr(), blocks, threads, iters,
                                int(bool(random_operands)), stream.cuda_stream), "cpk_mfma_loop")


def read_stream(src, out, blocks, stream):
    n16 = src.numel() * src.element_size() // 16
    if out.numel() < blocks * 256:
        raise ValueError("out holds fewer than blocks * 256 words")
    _check(load().cpk_read_stream(src.data_ptr(), n16, out.data_ptr(), blocks, stream.cuda_stream),
           "cpk_read_stream")
