"""Python binding of librkcalib (include/rk_calib.h): argument marshalling only.

Measured ceilings of the GPU (int32 VALU rate, copy and read bandwidth) for the
benchmark's roofline; the kernels run in the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librkcalib.so")
EXPORTS = ("rkc_valu_int32_rate", "rkc_copy_bandwidth", "rkc_read_bandwidth")

_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2307_01236_amd.build.build()")
        import torch  # noqa: F401  (one HIP runtime in the process, torch's)
        lib = C.CDLL(LIB_PATH)
        lib.rkc_valu_int32_rate.argtypes = [C.c_int32, C.POINTER(C.c_double)]
        lib.rkc_copy_bandwidth.argtypes = [C.c_int64, C.POINTER(C.c_double)]
        lib.rkc_read_bandwidth.argtypes = [C.c_int64, C.POINTER(C.c_double)]
        for n in EXPORTS:
            getattr(lib, n).restype = C.c_int
        _lib = lib
    return _lib


def _call(name, *args):
    out = C.c_double(0.0)
    rc = getattr(load(), name)(*args, C.byref(out))
    if rc != 0:
        raise RuntimeError(f"{name} failed ({rc})")
    return out.value


def valu_int32_rate(iters: int = 1 << 14) -> float:
    """Sustained int32 lane operations per second (add and min chains)."""
    return _call("rkc_valu_int32_rate", int(iters))


def copy_bandwidth(nbytes: int = 1 << 30) -> float:
    """Sustained device copy bandwidth, bytes read plus written per second."""
    return _call("rkc_copy_bandwidth", int(nbytes))


def read_bandwidth(nbytes: int = 1 << 30) -> float:
    """Sustained device read bandwidth, bytes read per second."""
    return _call("rkc_read_bandwidth", int(nbytes))
