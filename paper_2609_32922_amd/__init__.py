"""MI355X (gfx950) emulated stochastic-computing GEMM.

The product is libscgemm.so (C ABI in include/scgemm.h, HIP kernels in csrc/).
This package is its thin Python binding: ``_lib`` mirrors the C functions one to
one (same names), and ``gemm`` below only shapes torch device tensors into a
descriptor and calls ``sc_gemm``.  PyTorch supplies device memory and the stream;
every step of the computation runs in the library's kernels, and nothing falls
back to the CPU: without the built library every call raises.
"""
from __future__ import annotations

from ._lib import (SC_BIPOLAR_XNOR, SC_ERR_DEVICE_STATUS, SC_ERR_RESERVED, SC_KL_LIMIT, SC_NOALLOC_WORKSPACE_BYTES,  # noqa: F401
                   SC_L_MAX_LIMIT, SC_OK, SC_RNG_LFSR32, SC_RNG_SOBOL8_CBSG, SC_UNIPOLAR_AND_SM,
                   ScError, ScGemmDesc, load, sc_comparator_sequence, sc_gemm, sc_gemm_noalloc, sc_gemm_status,
                   sc_gemm_workspace_size, sc_mp_lengths, sc_quantize, sc_version, strerror)

__all__ = ["gemm", "make_desc", "comparator_sequence", "quantize", "mp_lengths", "Workspace",
           "ScGemmDesc", "ScError", "sc_gemm", "sc_gemm_noalloc", "sc_gemm_workspace_size", "sc_gemm_status",
           "sc_comparator_sequence", "sc_quantize", "sc_mp_lengths", "SC_BIPOLAR_XNOR",
           "SC_UNIPOLAR_AND_SM", "SC_RNG_LFSR32", "SC_RNG_SOBOL8_CBSG"]


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def make_desc(A, B, L_max: int, polarity: int, seed: int, L_hint: int = 0,
              rng: int = SC_RNG_LFSR32) -> ScGemmDesc:
    """Descriptor for contiguous A [batch, M, K] and B [batch or 1, N, K] tensors."""
    if A.dim() == 2:
        A = A.unsqueeze(0)
    if B.dim() == 2:
        B = B.unsqueeze(0)
    batch, M, K = A.shape
    nb, N, K2 = B.shape
    if K2 != K or nb not in (1, batch):
        raise ValueError("A is [batch, M, K], B must be [batch or 1, N, K]")
    d = ScGemmDesc()
    d.batch, d.M, d.N, d.K = batch, M, N, K
    d.lda, d.ldb, d.ldo = K, K, N
    d.strideA, d.strideB, d.strideO = M * K, (N * K if nb == batch and batch > 1 else 0), M * N
    d.strideSA, d.strideSB, d.strideL = M, (N if nb == batch and batch > 1 else 0), M
    d.L_max, d.polarity, d.rng, d.L_hint, d.seed = int(L_max), int(polarity), int(rng), int(L_hint), int(seed)
    return d


class Workspace:
    """A reusable device workspace (a torch uint8 tensor, 256-byte aligned)."""

    def __init__(self, nbytes: int, device="cuda"):
        import torch
        self.nbytes = int(nbytes)
        self._buf = torch.empty(self.nbytes + 256, dtype=torch.uint8, device=device)
        base = self._buf.data_ptr()
        self.ptr = (base + 255) // 256 * 256

    def ensure(self, nbytes: int):
        if nbytes > self.nbytes:
            self.__init__(nbytes, self._buf.device)
        return self


def _check_output(t, name, dtype, shape, device):
    """A caller-supplied output must be exactly what the kernels write into."""
    import torch
    if t.dtype != dtype:
        raise TypeError("%s must be %s, not %s" % (name, dtype, t.dtype))
    if not t.is_cuda or t.device != device:
        raise ValueError("%s must be on %s" % (name, device))
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor of shape %s, got %s" % (
            name, dtype, tuple(shape), tuple(t.shape)))
    return t


def gemm(A, sA, B, sB, L, *, L_max: int, polarity: int = SC_BIPOLAR_XNOR, seed: int = 0,
         out=None, counts=None, want_counts: bool = False, workspace: Workspace = None,
         stream=None, check_status: bool = False, prof_events=None, L_hint: int = 0,
         rng: int = SC_RNG_LFSR32):
    """SC GEMM on torch device tensors.

    A int8 [batch, M, K] (or [M, K]), sA float32 [batch, M], B int8 [batch or 1, N, K],
    sB float32 [batch or 1, N], L int32 [batch, M], all on one device.  ``rng`` selects
    the comparator source (LFSR, or Sobol-8 with conditional generation of B,
    L_max <= 256).  ``out`` (float32) and ``counts`` (int32), when given, must be
    contiguous [batch, M, N] tensors ([M, N] for 2-d A) on A's device.  When ``stream`` is
    not the current stream, tensors allocated here are marked as used by ``stream``.
    Returns (out, counts or None).
    """
    import torch
    squeeze = A.dim() == 2
    A3 = A.unsqueeze(0) if A.dim() == 2 else A
    B3 = B.unsqueeze(0) if B.dim() == 2 else B
    d = make_desc(A3, B3, L_max, polarity, seed, L_hint, rng)
    dev = A3.device
    for t, name in ((A3, "A"), (B3, "B"), (sA, "sA"), (sB, "sB"), (L, "L")):
        if not t.is_cuda or not t.is_contiguous() or t.device != dev:
            raise ValueError("%s must be a contiguous tensor on %s" % (name, dev))
    if A3.dtype != torch.int8 or B3.dtype != torch.int8 or sA.dtype != torch.float32 \
            or sB.dtype != torch.float32 or L.dtype != torch.int32:
        raise TypeError("dtypes: A, B int8; sA, sB float32; L int32")
    batch, M, N = d.batch, d.M, d.N
    if sA.numel() != batch * M or L.numel() != batch * M or sB.numel() != B3.shape[0] * N:
        raise ValueError("scale or length vector has the wrong size")
    oshape = (M, N) if squeeze else (batch, M, N)
    s = stream if stream is not None else torch.cuda.current_stream(dev)
    foreign = s != torch.cuda.current_stream(dev)
    made = []
    if out is None:
        out = torch.empty(oshape, dtype=torch.float32, device=dev)
        made.append(out)
    else:
        _check_output(out, "out", torch.float32, oshape, dev)
    if counts is None and want_counts:
        counts = torch.empty(oshape, dtype=torch.int32, device=dev)
        made.append(counts)
    elif counts is not None:
        _check_output(counts, "counts", torch.int32, oshape, dev)
    nbytes = sc_gemm_workspace_size(d)
    if workspace is None:
        ws = Workspace(nbytes, dev)
        made.append(ws._buf)
    else:
        ws = workspace.ensure(nbytes)
    if foreign:
        # the caching allocator must not hand these blocks out again before `s` is done
        for t in made:
            t.record_stream(s)
    if prof_events is not None:
        d.prof_event_begin = prof_events[0]
        d.prof_event_end = prof_events[1]
    sh = int(s.cuda_stream)
    rc = sc_gemm(d, A3.data_ptr(), sA.data_ptr(), B3.data_ptr(), sB.data_ptr(), L.data_ptr(),
                 out.data_ptr(), counts.data_ptr() if counts is not None else 0, ws.ptr, ws.nbytes, sh)
    if rc != SC_OK:
        raise ScError(rc, "sc_gemm")
    if check_status:
        rc = sc_gemm_status(ws.ptr, sh)
        if rc != SC_OK:
            raise ScError(rc, "sc_gemm (device status)")
    return out, counts


def comparator_sequence(seed: int, op: int, n: int, stream=None, rng: int = SC_RNG_LFSR32):
    """Device comparator sequence r_0..r_{n-1} (uint8 tensor) of operand ``op``."""
    import torch
    out = torch.empty(n, dtype=torch.uint8, device="cuda")
    rc = sc_comparator_sequence(seed, op, rng, n, out.data_ptr(), _stream_handle(stream))
    if rc != SC_OK:
        raise ScError(rc, "sc_comparator_sequence")
    return out


def quantize(X, per_tensor: bool = False, want_rowmax: bool = False, stream=None):
    """Device int8 quantisation of fp32 X [batch, rows, K] (or [rows, K]).

    Returns (Q int8, scale float32 [batch, rows], rowmax float32 or None).
    """
    import torch
    squeeze = X.dim() == 2
    X3 = X.unsqueeze(0) if squeeze else X
    if not X3.is_cuda or not X3.is_contiguous() or X3.dtype != torch.float32:
        raise ValueError("X must be a contiguous float32 device tensor")
    batch, rows, K = X3.shape
    Q = torch.empty((batch, rows, K), dtype=torch.int8, device=X.device)
    scale = torch.empty((batch, rows), dtype=torch.float32, device=X.device)
    rowmax = torch.empty((batch, rows), dtype=torch.float32, device=X.device) if want_rowmax else None
    rc = sc_quantize(batch, rows, K, X3.data_ptr(), K, rows * K, int(per_tensor), Q.data_ptr(), K,
                     rows * K, scale.data_ptr(), rowmax.data_ptr() if rowmax is not None else 0,
                     rows, _stream_handle(stream))
    if rc != SC_OK:
        raise ScError(rc, "sc_quantize")
    if squeeze:
        return Q[0], scale[0], (rowmax[0] if rowmax is not None else None)
    return Q, scale, rowmax


def mp_lengths(metric, tau, ladder, stream=None):
    """Per-row stream lengths (int32 device tensor shaped like ``metric``) from a row
    metric [batch, M] (or [M]) with thresholds ``tau`` and length ladder ``ladder``."""
    import torch
    squeeze = metric.dim() == 1
    m2 = metric.unsqueeze(0) if squeeze else metric
    if not m2.is_cuda or not m2.is_contiguous() or m2.dtype != torch.float32:
        raise ValueError("metric must be a contiguous float32 device tensor")
    batch, M = m2.shape
    L = torch.empty((batch, M), dtype=torch.int32, device=metric.device)
    rc = sc_mp_lengths(batch, M, m2.data_ptr(), M, list(tau), list(ladder), L.data_ptr(), M,
                       _stream_handle(stream))
    if rc != SC_OK:
        raise ScError(rc, "sc_mp_lengths")
    return L[0] if squeeze else L
