"""Pins of the oracle's front end: int8 quantisation and per-row length policy (CPU)."""
import numpy as np
import pytest

import workloads as W


def test_quantize_rows_closed_forms(oracle_mod):
    rng = np.random.default_rng(0)
    X = (rng.standard_normal((20, 37)) * rng.uniform(0.01, 10, (20, 1))).astype(np.float32)
    X[3] = 0.0
    Q, s, m = oracle_mod.quantize_rows_fp32(X)
    assert s[3] == 0 and m[3] == 0 and not Q[3].any()
    for i in range(20):
        if i == 3:
            continue
        assert m[i] == np.abs(X[i]).max()
        j = int(np.argmax(np.abs(X[i])))
        assert abs(int(Q[i, j])) == 127 and np.sign(Q[i, j]) == np.sign(X[i, j])
        # half a quantisation step at most (plus fp32 rounding of the scale)
        assert np.all(np.abs(Q[i].astype(np.float64) * s[i] - X[i]) <= 0.5 * s[i] * (1 + 1e-5))
    Qn, sn, _ = oracle_mod.quantize_rows_fp32(-X)
    assert np.array_equal(Qn, -Q) and np.array_equal(sn, s)


def test_quantize_grid_and_ties(oracle_mod):
    # integers on an exact power-of-two grid come back unchanged; halves round to even
    k = np.arange(-127, 128, dtype=np.float32)
    X = (k * np.float32(0.25))[None, :]
    Q, s, _ = oracle_mod.quantize_rows_fp32(X)
    assert s[0] == np.float32(31.75) / np.float32(127) and np.array_equal(Q[0], k.astype(np.int8))
    X = np.array([[127.0, 2.5, 3.5, -2.5, -3.5, 0.5, 1.5]], np.float32)
    Q, s, _ = oracle_mod.quantize_rows_fp32(X)
    assert s[0] == 1.0 and Q[0].tolist() == [127, 2, 4, -2, -4, 0, 2]


def test_quantize_matches_independent_host_quantiser(oracle_mod):
    rng = np.random.default_rng(1)
    X = rng.standard_normal((30, 50)).astype(np.float32)
    X[:, 7] *= 25
    Q, s, _ = oracle_mod.quantize_rows_fp32(X)
    Qw, sw = W.quantize_rows(X)
    assert np.array_equal(Q, Qw) and np.array_equal(s, sw)
    Qt, st = oracle_mod.quantize_tensor_fp32(X)
    Qtw, stw = W.quantize_tensor(X)
    assert np.array_equal(Qt, Qtw) and np.array_equal(st, stw)


def test_mp_lengths_definition(oracle_mod):
    ladder = [256, 192, 128, 64]
    tau = [0.75, 0.5, 0.25]
    g = np.array([0.0, 1.0, 0.25, 0.5, 0.75, 0.2499, 0.8, 0.1], np.float32)
    L = oracle_mod.mp_lengths_fp32(g, tau, ladder)
    assert L.tolist() == [64, 256, 128, 192, 256, 64, 256, 64]
    # min-max normalisation: an affine change of the metric changes nothing
    L2 = oracle_mod.mp_lengths_fp32(np.float32(3.0) * g + np.float32(5.0), tau, ladder)
    assert L2.tolist() == L.tolist()
    # a constant metric normalises to 0: every row gets the shortest length
    assert oracle_mod.mp_lengths_fp32(np.full(5, 2.0, np.float32), tau, ladder).tolist() == [64] * 5
    # one level: every row gets it
    assert oracle_mod.mp_lengths_fp32(g, [], [100]).tolist() == [100] * len(g)


def test_mp_lengths_monotone_and_quantile_thresholds(oracle_mod):
    # thresholds at the metric's quantiles reproduce the level counts they were fitted to
    rng = np.random.default_rng(2)
    g = rng.gamma(2.0, 1.0, 4001).astype(np.float32)
    ladder = [192, 96, 48, 24]
    counts = [400, 1000, 1601, 1000]
    t = (g - g.min()) / (g.max() - g.min())
    srt = np.sort(t)[::-1]
    tau = [float(srt[sum(counts[:k + 1]) - 1]) for k in range(3)]
    L = oracle_mod.mp_lengths_fp32(g, tau, ladder)
    assert [int((L == v).sum()) for v in ladder] == counts
    order = np.argsort(g, kind="stable")
    assert np.all(np.diff(L[order]) >= 0)
