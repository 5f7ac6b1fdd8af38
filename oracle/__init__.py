"""CPU oracle for emulated stochastic-computing matrix multiplication.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product library
(``paper_2609_32922_amd``) never imports it and shares no code with it.

The arithmetic lives in ``sc_oracle.c`` (plain C, OpenMP over rows, one byte per
stream bit, float64 decode); this module only builds it with gcc and marshals
numpy arrays through ctypes.  Each C function's header comment cites the passage
of the paper it follows (Sec. 3.1 encoding / comparator / Eq. (1), Sec. 4.2
boundaries and row lengths, Sec. A.1 LFSR).  The front-end functions at the end
(int8 quantisation, Sec. 3.1; per-row length policy, Sec. 4.4) are plain numpy
written element by element in fp32, the precision both sides take those integer
decisions in.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sc_oracle.c")
_LIB = os.path.join(_HERE, "libsc_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile ``sc_oracle.c`` into ``libsc_oracle.so`` with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                        _SRC, "-o", tmp], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        i32, u32, u64, vp = ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_void_p
        lib.oracle_splitmix64.argtypes = [u64]
        lib.oracle_splitmix64.restype = u64
        lib.oracle_seed_state.argtypes = [u64, u32]
        lib.oracle_seed_state.restype = u32
        lib.oracle_lfsr_draws.argtypes = [u32, i32, vp]
        lib.oracle_lfsr_draws.restype = None
        lib.oracle_lfsr_states.argtypes = [u32, i32, vp]
        lib.oracle_lfsr_states.restype = None
        lib.oracle_beta_bipolar.argtypes = [i32]
        lib.oracle_beta_bipolar.restype = i32
        lib.oracle_beta_unipolar.argtypes = [i32]
        lib.oracle_beta_unipolar.restype = i32
        lib.oracle_streams.argtypes = [i32, i32, vp, i32, u64, u32, i32, vp]
        lib.oracle_streams.restype = None
        lib.oracle_sc_gemm.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, u64,
                                       vp, vp, i32]
        lib.oracle_sc_gemm.restype = ctypes.c_int
        lib.oracle_sobol_shift.argtypes = [u64, u32]
        lib.oracle_sobol_shift.restype = u32
        lib.oracle_sobol8.argtypes = [ctypes.c_int, u32, i32, vp]
        lib.oracle_sobol8.restype = ctypes.c_int
        lib.oracle_sc_gemm_cbsg.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, u64,
                                            vp, vp, i32]
        lib.oracle_sc_gemm_cbsg.restype = ctypes.c_int
        lib.oracle_max_threads.argtypes = []
        lib.oracle_max_threads.restype = i32
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def splitmix64(x: int) -> int:
    return int(_load().oracle_splitmix64(ctypes.c_uint64(x & (2**64 - 1))))


def seed_state(seed: int, op: int) -> int:
    """Initial LFSR state of operand ``op`` (0 = A, 1 = B) for ``seed``."""
    return int(_load().oracle_seed_state(seed, op))


def lfsr_draws(state: int, n: int) -> np.ndarray:
    """``n`` comparator draws (uint8) from an initial LFSR state."""
    out = np.zeros(max(n, 1), np.uint8)
    _load().oracle_lfsr_draws(state, n, _ptr(out))
    return out[:n]


def lfsr_states(state: int, n: int) -> np.ndarray:
    out = np.zeros(max(n, 1), np.uint32)
    _load().oracle_lfsr_states(state, n, _ptr(out))
    return out[:n]


def comparator_sequence(seed: int, op: int, n: int) -> np.ndarray:
    """The comparator sequence r_0..r_{n-1} of operand ``op`` for ``seed``."""
    return lfsr_draws(seed_state(seed, op), n)


def beta_bipolar(q: int) -> int:
    return int(_load().oracle_beta_bipolar(int(q)))


def beta_unipolar(q: int) -> int:
    return int(_load().oracle_beta_unipolar(int(q)))


def streams(X: np.ndarray, polarity: int, seed: int, op: int, length: int) -> np.ndarray:
    """Materialised 0/1 streams, shape (rows, K, length), uint8."""
    X = np.ascontiguousarray(X, dtype=np.int8)
    rows, K = X.shape
    z = np.zeros((rows, K, max(length, 1)), np.uint8)
    _load().oracle_streams(rows, K, _ptr(X), polarity, seed, op, length, _ptr(z))
    return z[:, :, :length]


def sc_gemm(A: np.ndarray, B: np.ndarray, sA: np.ndarray, sB: np.ndarray,
            L: np.ndarray, L_max: int, polarity: int, seed: int,
            nthreads: int = 0, want_out: bool = True):
    """Oracle SC GEMM.  Returns ``(counts int32 MxN, out float64 MxN or None)``."""
    A = np.ascontiguousarray(A, dtype=np.int8)
    B = np.ascontiguousarray(B, dtype=np.int8)
    sA = np.ascontiguousarray(sA, dtype=np.float32)
    sB = np.ascontiguousarray(sB, dtype=np.float32)
    L = np.ascontiguousarray(L, dtype=np.int32)
    M, K = A.shape
    N, K2 = B.shape
    if K2 != K or sA.shape != (M,) or sB.shape != (N,) or L.shape != (M,):
        raise ValueError("shape mismatch")
    counts = np.zeros((M, N), np.int32)
    out = np.zeros((M, N), np.float64) if want_out else None
    rc = _load().oracle_sc_gemm(M, N, K, _ptr(A), _ptr(B), _ptr(sA), _ptr(sB), _ptr(L),
                                int(L_max), int(polarity), ctypes.c_uint64(seed),
                                _ptr(counts), _ptr(out), int(nthreads))
    if rc != 0:
        raise ValueError("oracle_sc_gemm failed with code %d" % rc)
    return counts, out


def decode(counts: np.ndarray, sA: np.ndarray, sB: np.ndarray, L: np.ndarray, K: int,
           polarity: int) -> np.ndarray:
    """Eq. (1) (Sec. 3.1, "SC matrix multiplication") applied to a count matrix, float64.

    counts [M, N] int: X_ij (bipolar XNOR counts) or S_ij (unipolar signed AND counts).
    Bipolar  out_ij = sA_i sB_j 127^2 (2 X_ij / L_i - K); unipolar out_ij = sA_i sB_j 127^2
    S_ij / L_i; a row with L_i = 0 decodes to 0.  The same formula, in the same order of
    operations, as the decode inside ``sc_gemm``, written out element-wise in numpy so it
    can be applied to any count matrix.
    """
    c = np.asarray(counts, dtype=np.float64)
    M, N = c.shape
    a = np.asarray(sA, dtype=np.float32).astype(np.float64).reshape(M, 1)
    b = np.asarray(sB, dtype=np.float32).astype(np.float64).reshape(1, N)
    Li = np.asarray(L, dtype=np.int64).reshape(M, 1)
    scale = a * b * float(127 * 127)
    Ld = np.where(Li > 0, Li, 1).astype(np.float64)
    if polarity == 0:
        out = scale * (2.0 * c / Ld - float(K))
    else:
        out = scale * c / Ld
    return np.where(Li > 0, out, 0.0)


def sobol_shift(seed: int, op: int) -> int:
    return int(_load().oracle_sobol_shift(ctypes.c_uint64(seed), op))


def sobol8(dim: int, shift: int, n: int = 256) -> np.ndarray:
    """First n (<= 256) points of scrambled Sobol-8 dimension ``dim`` (1 or 2), uint8."""
    out = np.zeros(max(n, 1), np.uint8)
    if _load().oracle_sobol8(dim, shift, n, _ptr(out)) != 0:
        raise ValueError("bad Sobol arguments")
    return out[:n]


def sc_gemm_cbsg(A: np.ndarray, B: np.ndarray, sA: np.ndarray, sB: np.ndarray,
                 L: np.ndarray, L_max: int, polarity: int, seed: int,
                 nthreads: int = 0, want_out: bool = True):
    """Oracle SC GEMM with Sobol-8 C-BSG streams.  Returns (counts, out)."""
    A = np.ascontiguousarray(A, dtype=np.int8)
    B = np.ascontiguousarray(B, dtype=np.int8)
    sA = np.ascontiguousarray(sA, dtype=np.float32)
    sB = np.ascontiguousarray(sB, dtype=np.float32)
    L = np.ascontiguousarray(L, dtype=np.int32)
    M, K = A.shape
    N, K2 = B.shape
    if K2 != K or sA.shape != (M,) or sB.shape != (N,) or L.shape != (M,):
        raise ValueError("shape mismatch")
    counts = np.zeros((M, N), np.int32)
    out = np.zeros((M, N), np.float64) if want_out else None
    rc = _load().oracle_sc_gemm_cbsg(M, N, K, _ptr(A), _ptr(B), _ptr(sA), _ptr(sB), _ptr(L),
                                     int(L_max), int(polarity), ctypes.c_uint64(seed),
                                     _ptr(counts), _ptr(out), int(nthreads))
    if rc != 0:
        raise ValueError("oracle_sc_gemm_cbsg failed with code %d" % rc)
    return counts, out


def max_threads() -> int:
    return int(_load().oracle_max_threads())


# ----------------------------------------------------------------------------
# front end: symmetric int8 quantisation and the per-row length policy
# (plain numpy, row by row, IEEE fp32 as the device computes it)
# ----------------------------------------------------------------------------

def quantize_rows_fp32(X: np.ndarray):
    """Per-row symmetric int8 quantisation (Sec. 3.1: s_i = max_d |X_id| / q_max).

    Returns (Q int8, s float32, m float32) with m_i = max_d |X_id|.  Every step is an
    fp32 operation: s = m / 127, Q = clamp(rint(x / s), -127, 127) (half to even);
    s = 0 gives Q = 0.
    """
    X = np.asarray(X, dtype=np.float32)
    rows, K = X.shape
    Q = np.zeros((rows, K), np.int8)
    s = np.zeros(rows, np.float32)
    m = np.zeros(rows, np.float32)
    for i in range(rows):
        mi = np.float32(0.0)
        for d in range(K):
            a = np.float32(abs(X[i, d]))
            if a > mi:
                mi = a
        m[i] = mi
        si = np.float32(mi / np.float32(127.0))
        s[i] = si
        if si > 0:
            q = np.rint(X[i] / si)                    # fp32 division, half-to-even
            Q[i] = np.clip(q, -127, 127).astype(np.int8)
    return Q, s, m


def quantize_tensor_fp32(X: np.ndarray):
    """Per-tensor symmetric int8 quantisation: one scale m/127 with m = max |X|."""
    X = np.asarray(X, dtype=np.float32)
    rows, K = X.shape
    m = np.float32(0.0)
    for i in range(rows):
        for d in range(K):
            a = np.float32(abs(X[i, d]))
            if a > m:
                m = a
    sc = np.float32(m / np.float32(127.0))
    Q = np.zeros((rows, K), np.int8)
    if sc > 0:
        for i in range(rows):
            Q[i] = np.clip(np.rint(X[i] / sc), -127, 127).astype(np.int8)
    return Q, np.full(rows, sc, np.float32)


def mp_lengths_fp32(metric: np.ndarray, tau, ladder) -> np.ndarray:
    """Per-row stream lengths of one operator call (Sec. 4.4).

    t_i = (g_i - min g) / (max g - min g) in fp32 (0 when max = min); row i gets
    ladder[k] for the first k with t_i >= tau[k], else the shortest, ladder[-1].
    """
    g = np.asarray(metric, dtype=np.float32)
    lo = np.float32(g.min()) if g.size else np.float32(0)
    hi = np.float32(g.max()) if g.size else np.float32(0)
    rng = np.float32(hi - lo)
    out = np.zeros(g.shape[0], np.int32)
    for i in range(g.shape[0]):
        t = np.float32(np.float32(g[i] - lo) / rng) if rng > 0 else np.float32(0.0)
        k = len(ladder) - 1
        for j in range(len(ladder) - 1):
            if t >= np.float32(tau[j]):
                k = j
                break
        out[i] = int(ladder[k])
    return out
