"""ctypes binding of libscpeak (include/scpeak.h): the measured VALU rate of the packed
AND + popcount stream, which the benchmark reports beside the SC GEMM's rate.  Marshalling
only; loading fails loudly when the library has not been built."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libscpeak.so")


class ScPeakResult(ctypes.Structure):
    """Mirror of ``sc_peak_result``."""
    _fields_ = [
        ("seconds", ctypes.c_double),
        ("lane_ops_per_s", ctypes.c_double),
        ("bitops_per_s", ctypes.c_double),
        ("clock_hz", ctypes.c_double),
        ("cus", ctypes.c_int32),
        ("waves_per_simd", ctypes.c_int32),
    ]


_lib = None


def load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libscpeak.so is not built (%s); run python -m paper_2609_32922_amd.build"
                              % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        lib.sc_peak_valu_bitop.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ScPeakResult)]
        lib.sc_peak_valu_bitop.restype = ctypes.c_int
        _lib = lib
    return _lib


def sc_peak_valu_bitop(waves_per_simd: int, iters: int) -> ScPeakResult:
    r = ScPeakResult()
    rc = load().sc_peak_valu_bitop(int(waves_per_simd), int(iters), ctypes.byref(r))
    if rc != 0:
        raise RuntimeError("sc_peak_valu_bitop failed with code %d" % rc)
    return r
