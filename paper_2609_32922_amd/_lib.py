"""ctypes binding of libscgemm (the C ABI declared in include/scgemm.h).

Argument marshalling only: every step of the SC GEMM runs in the library's HIP
kernels.  Loading fails loudly when the built library is missing; there is no
fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libscgemm.so")

SC_OK = 0
SC_ERR_NULL = -1
SC_ERR_SHAPE = -2
SC_ERR_LEN = -3
SC_ERR_POLARITY = -4
SC_ERR_RNG = -5
SC_ERR_WORKSPACE = -6
SC_ERR_HIP = -7
SC_ERR_DEVICE_STATUS = -8
SC_ERR_STRIDE = -9
SC_ERR_RESERVED = -10

SC_BIPOLAR_XNOR = 0
SC_UNIPOLAR_AND_SM = 1
SC_RNG_LFSR32 = 0
SC_RNG_SOBOL8_CBSG = 1
SC_L_MAX_LIMIT = 4096
SC_K_LIMIT = 1 << 20
SC_KL_LIMIT = 1 << 27
SC_NOALLOC_WORKSPACE_BYTES = 64 << 20


class ScGemmDesc(ctypes.Structure):
    """Mirror of ``sc_gemm_desc`` (field order and types as in scgemm.h)."""
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("M", ctypes.c_int32),
        ("N", ctypes.c_int32),
        ("K", ctypes.c_int32),
        ("lda", ctypes.c_int64),
        ("ldb", ctypes.c_int64),
        ("ldo", ctypes.c_int64),
        ("strideA", ctypes.c_int64),
        ("strideB", ctypes.c_int64),
        ("strideO", ctypes.c_int64),
        ("strideSA", ctypes.c_int64),
        ("strideSB", ctypes.c_int64),
        ("strideL", ctypes.c_int64),
        ("L_max", ctypes.c_int32),
        ("polarity", ctypes.c_int32),
        ("rng", ctypes.c_int32),
        ("L_hint", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("prof_event_begin", ctypes.c_void_p),
        ("prof_event_end", ctypes.c_void_p),
    ]


class ScError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__("%s failed: %s (%d)" % (where, strerror(code), code))


_lib = None


def load():
    """Load libscgemm.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libscgemm.so is not built (%s); run __graft_entry__.build() or "
            "python -m paper_2609_32922_amd.build" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    pdesc = ctypes.POINTER(ScGemmDesc)
    lib.sc_gemm_workspace_size.argtypes = [pdesc, ctypes.POINTER(sz)]
    lib.sc_gemm_workspace_size.restype = ctypes.c_int
    lib.sc_gemm.argtypes = [pdesc, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.sc_gemm.restype = ctypes.c_int
    lib.sc_gemm_noalloc.argtypes = [pdesc, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.sc_gemm_noalloc.restype = ctypes.c_int
    lib.sc_gemm_status.argtypes = [vp, vp]
    lib.sc_gemm_status.restype = ctypes.c_int
    lib.sc_comparator_sequence.argtypes = [u64, i32, i32, i32, vp, vp]
    lib.sc_comparator_sequence.restype = ctypes.c_int
    f32p = ctypes.POINTER(ctypes.c_float)
    i32p = ctypes.POINTER(ctypes.c_int32)
    i64 = ctypes.c_int64
    lib.sc_quantize.argtypes = [i32, i32, i32, vp, i64, i64, i32, vp, i64, i64, vp, vp, i64, vp]
    lib.sc_quantize.restype = ctypes.c_int
    lib.sc_mp_lengths.argtypes = [i32, i32, vp, i64, f32p, i32p, i32, vp, i64, vp]
    lib.sc_mp_lengths.restype = ctypes.c_int
    lib.sc_strerror.argtypes = [ctypes.c_int]
    lib.sc_strerror.restype = ctypes.c_char_p
    lib.sc_version.argtypes = []
    lib.sc_version.restype = ctypes.c_int
    _lib = lib
    return lib


def strerror(code: int) -> str:
    return load().sc_strerror(int(code)).decode()


def sc_gemm_workspace_size(desc: ScGemmDesc) -> int:
    n = ctypes.c_size_t(0)
    rc = load().sc_gemm_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    if rc != SC_OK:
        raise ScError(rc, "sc_gemm_workspace_size")
    return int(n.value)


def sc_gemm(desc: ScGemmDesc, A: int, sA: int, B: int, sB: int, L_per_row: int, out: int,
            counts: int, workspace: int, workspace_bytes: int, stream: int) -> int:
    """Raw call with integer device addresses; returns the status code."""
    return int(load().sc_gemm(ctypes.byref(desc), A, sA, B, sB, L_per_row, out, counts or None,
                              workspace, workspace_bytes, stream or None))


def sc_gemm_noalloc(desc: ScGemmDesc, A: int, sA: int, B: int, sB: int, L_per_row: int, out: int,
                    counts: int, status_out: int, stream: int) -> int:
    """Raw call of the allocation-free entry point (the library's own static workspace)."""
    return int(load().sc_gemm_noalloc(ctypes.byref(desc), A, sA, B, sB, L_per_row, out, counts or None,
                                      status_out or None, stream or None))


def sc_gemm_status(workspace: int, stream: int) -> int:
    return int(load().sc_gemm_status(workspace, stream or None))


def sc_comparator_sequence(seed: int, op: int, rng: int, n: int, out: int, stream: int) -> int:
    return int(load().sc_comparator_sequence(ctypes.c_uint64(seed), op, rng, n, out, stream or None))


def sc_quantize(batch: int, rows: int, K: int, X: int, ldx: int, strideX: int, per_tensor: int,
                Q: int, ldq: int, strideQ: int, scale: int, rowmax: int, strideS: int,
                stream: int) -> int:
    return int(load().sc_quantize(batch, rows, K, X, ldx, strideX, per_tensor, Q, ldq, strideQ,
                                  scale, rowmax or None, strideS, stream or None))


def sc_mp_lengths(batch: int, M: int, metric: int, strideM: int, tau, ladder, L_out: int,
                  strideL: int, stream: int) -> int:
    n = len(ladder)
    tau_a = (ctypes.c_float * max(len(tau), 1))(*[float(x) for x in tau])
    lad_a = (ctypes.c_int32 * max(n, 1))(*[int(x) for x in ladder])
    return int(load().sc_mp_lengths(batch, M, metric, strideM, tau_a, lad_a, n, L_out, strideL,
                                    stream or None))


def sc_version() -> int:
    return int(load().sc_version())
