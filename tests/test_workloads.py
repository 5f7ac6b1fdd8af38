"""Seeded input generators: determinism, quantisation and length budgets (CPU only)."""
import numpy as np
import pytest

import workloads as W


def test_quantize_rows_definition():
    rng = np.random.default_rng(0)
    X = rng.standard_normal((5, 33)).astype(np.float32)
    X[2] = 0.0
    q, s = W.quantize_rows(X)
    assert q.dtype == np.int8 and s.dtype == np.float32
    assert s[2] == 0 and not q[2].any()
    for i in (0, 1, 3, 4):
        m = np.abs(X[i]).max()
        assert s[i] == np.float32(m / np.float32(127))
        assert np.abs(q[i]).max() == 127
        assert np.all(np.abs(q[i].astype(np.float32) * s[i] - X[i]) <= 0.5 * s[i] * (1 + 1e-6))


@pytest.mark.parametrize("lo,hi,mean", [(16, 256, 64), (8, 512, 96), (8, 512, 128)])
def test_lengths_matched_mean(lo, hi, mean):
    rng = np.random.default_rng(lo + hi)
    g = np.abs(rng.standard_normal(3001)) + 0.1
    L = W.lengths_matched_mean(g, lo, hi, mean)
    assert L.sum() == mean * len(g)
    assert L.min() >= lo and L.max() <= hi
    # monotone in the metric up to the rounding unit
    order = np.argsort(g)
    assert np.all(np.diff(L[order]) >= -1)


def test_workloads_deterministic_and_shaped():
    w1 = W.bipolar_64x256x64()
    w2 = W.bipolar_64x256x64()
    g1, g2 = w1.gemms[0], w2.gemms[0]
    assert np.array_equal(g1.A, g2.A) and np.array_equal(g1.B, g2.B)
    assert g1.A.shape == (1, 64, 256) and g1.B.shape == (1, 64, 256)
    assert w1.bitops() == 64 * 64 * 256 * 64
    w = W.ditxl2_proj_mlp_group96()
    for g in w.gemms:
        Lg = g.L[0].reshape(-1, 32)
        assert np.all(Lg == Lg[:, :1])                    # constant per group of 32
        assert sorted(set(Lg[:, 0].tolist())) == [24, 48, 96, 192]
        assert g.L.sum() == 96 * 4096
    assert w.bitops() == 4096 * 1152 * 96 * (3456 + 4608)
