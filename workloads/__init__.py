"""Seeded synthetic workloads for the SC GEMM (shared by the tests and the benchmark).

This module holds no stochastic-computing arithmetic: it only draws seeded random
tensors with the shapes and value distributions of the layers the paper evaluates,
applies the standard symmetric int8 post-training quantisation that the paper takes
as given before the SC matmul (Sec. 3.1 "SC matrix multiplication": per-row scales
s_i = max_d |X_id| / q_max, integers in [-q_max, q_max]), and assigns per-row stream
lengths.  Both the CPU oracle and the GPU library consume exactly these int8
matrices, scales and length vectors.

The paper's datasets and pretrained weights (ImageNet with DINOv2 ViT-L/14, COCO
with EVA-01, DiT-XL/2, Dino-WM) are not available, so every workload is synthetic:
random-init tensors with the real layer shapes (ViT-B/16 at 224 px, DiT-XL/2 at
256 px, ViT-L/14 at 336 px).  The row-length vectors stand in for the paper's
calibrated mixed-precision policy (Sec. 4.4): lengths proportional to the row's
max-abs metric, clamped, renormalised to a matched average.

Draw order is fixed; ``numpy.random.default_rng(seed)`` (PCG64) everywhere.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

QMAX = 127
BIPOLAR = 0
UNIPOLAR_SM = 1


@dataclass
class Gemm:
    """One SC GEMM problem: out[b] = decode(A[b] (M x K) . B[b]^T (N x K))."""
    name: str
    A: np.ndarray            # int8 [batch, M, K]
    sA: np.ndarray           # float32 [batch, M]
    B: np.ndarray            # int8 [batch or 1, N, K]
    sB: np.ndarray           # float32 [batch or 1, N]
    L: np.ndarray            # int32 [batch, M]
    L_max: int
    polarity: int
    seed: int

    @property
    def batch(self) -> int:
        return self.A.shape[0]

    @property
    def M(self) -> int:
        return self.A.shape[1]

    @property
    def N(self) -> int:
        return self.B.shape[1]

    @property
    def K(self) -> int:
        return self.A.shape[2]

    def bitops(self) -> int:
        """Algorithmic stream-bit-ops N * K * sum(L_i), over the whole batch."""
        return int(self.N) * int(self.K) * int(self.L.astype(np.int64).sum())


@dataclass
class Workload:
    name: str
    description: str
    gemms: List[Gemm] = field(default_factory=list)

    def bitops(self) -> int:
        return sum(g.bitops() for g in self.gemms)


# ----------------------------------------------------------------------------
# quantisation and length assignment (input preparation, not part of the path)
# ----------------------------------------------------------------------------

def quantize_rows(X: np.ndarray):
    """Symmetric int8 per-row quantisation: s = maxabs/127 (fp32), q = clamp(rint(x/s)).

    A zero row gets s = 0 and q = 0.  Division and rounding are IEEE fp32 with
    round-half-to-even, so the result is reproducible bit for bit.
    """
    X = np.asarray(X, dtype=np.float32)
    maxabs = np.max(np.abs(X), axis=-1).astype(np.float32)
    s = (maxabs / np.float32(QMAX)).astype(np.float32)
    safe = np.where(s > 0, s, np.float32(1.0)).astype(np.float32)
    q = np.rint(X / safe[..., None]).astype(np.float32)
    q = np.clip(q, -QMAX, QMAX)
    q = np.where(s[..., None] > 0, q, 0).astype(np.int8)
    return q, s


def quantize_tensor(X: np.ndarray):
    """Symmetric int8 per-tensor quantisation; the scale is broadcast to every row."""
    X = np.asarray(X, dtype=np.float32)
    maxabs = np.float32(np.max(np.abs(X)))
    s = np.float32(maxabs / np.float32(QMAX))
    safe = s if s > 0 else np.float32(1.0)
    q = np.clip(np.rint(X / safe), -QMAX, QMAX)
    q = (q if s > 0 else np.zeros_like(q)).astype(np.int8)
    return q, np.full(X.shape[:-1], s, np.float32)


def lengths_matched_mean(metric: np.ndarray, L_lo: int, L_hi: int, L_mean: int) -> np.ndarray:
    """Per-row lengths proportional to ``metric``, clamped to [L_lo, L_hi], sum = L_mean*M.

    Bisection on the proportionality constant c so that sum(clamp(c*g)) = L_mean*M,
    then floor, then hand out the remaining units by largest fractional part (ties
    to the lower index) among rows still below L_hi.  The sum is exact.
    """
    g = np.asarray(metric, dtype=np.float64)
    M = g.size
    target = int(L_mean) * M
    if not (L_lo * M <= target <= L_hi * M):
        raise ValueError("mean length outside the clamp range")
    gpos = np.maximum(g, 1e-30)
    lo, hi = 0.0, 1.0
    while np.clip(hi * gpos, L_lo, L_hi).sum() < target:
        hi *= 2.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if np.clip(mid * gpos, L_lo, L_hi).sum() < target:
            lo = mid
        else:
            hi = mid
    v = np.clip(hi * gpos, L_lo, L_hi)
    f = np.floor(v).astype(np.int64)
    rem = target - int(f.sum())
    if rem < 0:
        # hi overshoots by rounding: take units back from the largest rows above L_lo
        frac = v - f
        order = np.lexsort((np.arange(M), frac))
        for idx in order:
            if rem == 0:
                break
            if f[idx] > L_lo:
                f[idx] -= 1
                rem += 1
    else:
        frac = v - f
        order = np.lexsort((np.arange(M), -frac))
        for idx in order:
            if rem == 0:
                break
            if f[idx] < L_hi:
                f[idx] += 1
                rem -= 1
    assert rem == 0 and f.sum() == target
    return f.astype(np.int32)


def _heavy_tail_normal(rng: np.random.Generator, shape, frac: float = 0.01, df: float = 3.0):
    """N(0,1) with each entry replaced by a Student-t(df) draw with probability ``frac``."""
    x = rng.standard_normal(shape, dtype=np.float32)
    mask = rng.random(shape) < frac
    t = rng.standard_t(df, size=shape).astype(np.float32)
    return np.where(mask, t, x).astype(np.float32)


# ----------------------------------------------------------------------------
# the five workloads
# ----------------------------------------------------------------------------

def bipolar_64x256x64(seed: int = 0) -> Workload:
    """Single bipolar SC GEMM, M=64 K=256 N=64, L=64 for every row, comparator seed 0.

    A ~ U[-1,1], per-row scales; B ~ N(0, 0.02), per-tensor scale.
    """
    rng = np.random.default_rng(seed)
    M, K, N, L = 64, 256, 64, 64
    A = rng.uniform(-1.0, 1.0, (M, K)).astype(np.float32)
    B = (rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)).astype(np.float32)
    qA, sA = quantize_rows(A)
    qB, sB = quantize_tensor(B)
    g = Gemm("gemm", qA[None], sA[None], qB[None], sB[None],
             np.full((1, M), L, np.int32), L, BIPOLAR, seed)
    return Workload("bipolar_64x256x64_L64", "bipolar SC GEMM 64x256x64, uniform L=64", [g])


def _vitb_fc1_inputs(rng: np.random.Generator):
    M, K, N = 32 * 197, 768, 3072
    X = rng.standard_normal((M, K), dtype=np.float32)
    outl = rng.choice(K, 6, replace=False)
    X[:, outl] *= np.float32(20.0)
    W = (rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)).astype(np.float32)
    qA, sA = quantize_rows(X)
    qB, sB = quantize_tensor(W)
    return qA, sA, qB, sB, np.max(np.abs(X), axis=1)


def vitb16_fc1_L128(seed: int = 1) -> Workload:
    """ViT-B/16 MLP fc1 (batch 32 x 197 tokens): M=6304, K=768, N=3072, bipolar, L=128.

    Activations N(0,1) with 6 random outlier channels x20, per-row scales; weights
    N(0, 0.02), per-tensor scale.
    """
    rng = np.random.default_rng(seed)
    qA, sA, qB, sB, _ = _vitb_fc1_inputs(rng)
    M = qA.shape[0]
    g = Gemm("fc1", qA[None], sA[None], qB[None], sB[None],
             np.full((1, M), 128, np.int32), 128, BIPOLAR, seed)
    return Workload("vitb16_fc1_L128", "ViT-B/16 fc1 6304x768x3072, bipolar, uniform L=128", [g])


def vitb16_fc1_mp64(seed: int = 2) -> Workload:
    """ViT-B/16 fc1 under per-row lengths: L_i in [16,256] proportional to row max-abs,
    renormalised to mean 64; bipolar."""
    rng = np.random.default_rng(seed)
    qA, sA, qB, sB, gmet = _vitb_fc1_inputs(rng)
    L = lengths_matched_mean(gmet, 16, 256, 64)
    g = Gemm("fc1", qA[None], sA[None], qB[None], sB[None], L[None], 256, BIPOLAR, seed)
    return Workload("vitb16_fc1_mp64", "ViT-B/16 fc1 6304x768x3072, bipolar, per-row L in [16,256], mean 64", [g])


def ditxl2_proj_mlp_group96(seed: int = 3) -> Workload:
    """DiT-XL/2 attention projection (4096x1152x3456) and MLP (4096x1152x4608).

    Activations Laplace(0,1), per-row scales; weights N(0,0.02), per-tensor scale.
    Per-group lengths: 128 groups of 32 rows ranked by group max-abs, the top 40 get
    L=192, the next 24 get 96, the next 32 get 48 and the last 32 get 24 (mean 96).
    Unipolar AND, sign-magnitude.
    """
    rng = np.random.default_rng(seed)
    M, K = 16 * 256, 1152
    gemms = []
    for name, N in (("qkv_proj", 3456), ("mlp_fc1", 4608)):
        X = rng.laplace(0.0, 1.0, (M, K)).astype(np.float32)
        W = (rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)).astype(np.float32)
        qA, sA = quantize_rows(X)
        qB, sB = quantize_tensor(W)
        gmax = np.max(np.abs(X).reshape(M // 32, 32 * K), axis=1)
        order = np.lexsort((np.arange(M // 32), -gmax))   # descending metric, ties by index
        Lg = np.empty(M // 32, np.int32)
        ladder = [192] * 40 + [96] * 24 + [48] * 32 + [24] * 32
        Lg[order] = np.array(ladder, np.int32)
        L = np.repeat(Lg, 32).astype(np.int32)
        gemms.append(Gemm(name, qA[None], sA[None], qB[None], sB[None], L[None], 192,
                          UNIPOLAR_SM, seed))
    return Workload("ditxl2_proj_mlp_group96",
                    "DiT-XL/2 proj 4096x1152x3456 + MLP 4096x1152x4608, unipolar SM, per-group L mean 96",
                    gemms)


def vitl14_336_qk_mlp(seed: int = 4, qk: bool = True, mlp: bool = True) -> Workload:
    """ViT-L/14 at 336 px: attention Q.K^T (8 x 16 heads, 577 x 64) and MLP fc1
    (18464 x 1024 x 4096), bipolar, per-row lengths in [8,512] (means 96 and 128).

    Inputs N(0,1) with 1% heavy-tail Student-t(3) entries; Q, K and X per-row
    scales; W ~ N(0,0.02) per-tensor.  Q.K^T lengths follow ||Q_i||_inf per head,
    MLP lengths follow ||X_i||_inf.
    """
    rng = np.random.default_rng(seed)
    gemms = []
    H, S, Dh = 8 * 16, 577, 64
    Q = _heavy_tail_normal(rng, (H, S, Dh))
    Kt = _heavy_tail_normal(rng, (H, S, Dh))
    if qk:
        qQ, sQ = quantize_rows(Q)
        qK, sK = quantize_rows(Kt)
        L = np.stack([lengths_matched_mean(np.max(np.abs(Q[h]), axis=1), 8, 512, 96)
                      for h in range(H)])
        gemms.append(Gemm("attn_qk", qQ, sQ, qK, sK, L.astype(np.int32), 512, BIPOLAR, seed))
    M, K, N = 32 * 577, 1024, 4096
    X = _heavy_tail_normal(rng, (M, K))
    W = (rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)).astype(np.float32)
    if mlp:
        qX, sX = quantize_rows(X)
        qW, sW = quantize_tensor(W)
        L = lengths_matched_mean(np.max(np.abs(X), axis=1), 8, 512, 128)
        gemms.append(Gemm("mlp_fc1", qX[None], sX[None], qW[None], sW[None], L[None], 512,
                          BIPOLAR, seed))
    return Workload("vitl14_336_qk_mlp",
                    "ViT-L/14-336 QK^T 128x(577x64x577) mean L 96 + MLP 18464x1024x4096 mean L 128, bipolar",
                    gemms)


def vitl14_compensator_L256(seed: int = 5) -> Workload:
    """Per-head residual compensator of one ViT-L/14 block (224 px, batch 32 x 257 tokens):
    16 heads, each a 64x64 SC matmul of the head's slice of the block input, at the
    uniform compensator length L = 256, bipolar (Sec. A.2: W_b stored per head, the
    compensator itself an SC matmul at L_comp = 256).

    Block input x ~ N(0,1) with 1% Student-t(3) entries, per-row scales of each head's
    slice; W_h ~ N(0, 0.02), per-head per-tensor scale.
    """
    rng = np.random.default_rng(seed)
    T, H, dh = 32 * 257, 16, 64
    x = _heavy_tail_normal(rng, (T, H * dh))
    Wc = (rng.standard_normal((H, dh, dh), dtype=np.float32) * np.float32(0.02)).astype(np.float32)
    xs = np.ascontiguousarray(x.reshape(T, H, dh).transpose(1, 0, 2))     # [H, T, 64]
    qA, sA = quantize_rows(xs)
    qB = np.empty((H, dh, dh), np.int8)
    sB = np.empty((H, dh), np.float32)
    for h in range(H):
        qB[h], sB[h] = quantize_tensor(Wc[h])
    g = Gemm("compensator", qA, sA, qB, sB, np.full((H, T), 256, np.int32), 256, BIPOLAR, seed)
    return Workload("vitl14_compensator_L256",
                    "ViT-L/14 per-head compensator 16 x (8224x64x64), bipolar, L = 256", [g])


def vitl14_336_attn_av(seed: int = 6) -> Workload:
    """Attention probabilities times values, ViT-L/14 at 336 px: 8 x 16 heads of
    P (577 x 577, softmax rows, values in [0,1]) times V (577 x 64).  In the A.B^T form
    A = P (M = K = 577) and B = V^T (N = 64).  Unipolar sign-magnitude (P >= 0, V signed).
    Row lengths follow the peak attention probability max_j P_ij (Sec. 4.4 metric of the
    av operator), in [8, 512] with mean 96 per head.
    """
    rng = np.random.default_rng(seed)
    H, S, dh = 8 * 16, 577, 64
    Qm = _heavy_tail_normal(rng, (H, S, dh))
    Km = _heavy_tail_normal(rng, (H, S, dh))
    V = _heavy_tail_normal(rng, (H, S, dh))
    logits = np.einsum("hid,hjd->hij", Qm, Km, optimize=True).astype(np.float32) / np.float32(8.0)
    logits -= logits.max(axis=2, keepdims=True)
    P = np.exp(logits).astype(np.float32)
    P /= P.sum(axis=2, keepdims=True)
    qP, sP = quantize_rows(P)
    Vt = np.ascontiguousarray(V.transpose(0, 2, 1))                      # [H, 64, 577]
    qV, sV = quantize_rows(Vt)
    L = np.stack([lengths_matched_mean(P[h].max(axis=1), 8, 512, 96) for h in range(H)])
    g = Gemm("attn_av", qP, sP, qV, sV, L.astype(np.int32), 512, UNIPOLAR_SM, seed)
    return Workload("vitl14_336_attn_av",
                    "ViT-L/14-336 attention P.V 128 x (577x577x64), unipolar SM, per-row L mean 96", [g])


WORKLOADS: Dict[str, callable] = {
    "bipolar_64x256x64_L64": bipolar_64x256x64,
    "vitb16_fc1_L128": vitb16_fc1_L128,
    "vitb16_fc1_mp64": vitb16_fc1_mp64,
    "ditxl2_proj_mlp_group96": ditxl2_proj_mlp_group96,
    "vitl14_336_qk_mlp": vitl14_336_qk_mlp,
    "vitl14_compensator_L256": vitl14_compensator_L256,
    "vitl14_336_attn_av": vitl14_336_attn_av,
}


def random_gemm(rng: np.random.Generator, batch: int, M: int, N: int, K: int,
                L_max: int, polarity: int, seed: int, L_lo: int = 0,
                broadcast_B: bool = False, uniform_L: Optional[int] = None) -> Gemm:
    """A small random problem with uniformly random int8 entries and lengths."""
    A = rng.integers(-127, 128, (batch, M, K)).astype(np.int8)
    nb = 1 if broadcast_B else batch
    B = rng.integers(-127, 128, (nb, N, K)).astype(np.int8)
    sA = rng.uniform(0.001, 0.05, (batch, M)).astype(np.float32)
    sB = rng.uniform(0.001, 0.05, (nb, N)).astype(np.float32)
    if uniform_L is not None:
        L = np.full((batch, M), uniform_L, np.int32)
    else:
        L = rng.integers(L_lo, L_max + 1, (batch, M)).astype(np.int32)
    return Gemm("random", A, sA, B, sB, L, L_max, polarity, seed)
