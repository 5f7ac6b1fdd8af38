"""Pins of the oracle's Sobol-8 / C-BSG datapath (Sec. 4.2, Sec. A.1) -- CPU only."""
from fractions import Fraction

import numpy as np
import pytest

import sc_bruteforce as bf


def test_sobol_direction_numbers_published():
    # dimension 2 (primitive polynomial x + 1): m = 1, 3, 5, 15, 17, 51, 85, 255
    m = [1]
    for _ in range(7):
        m.append((2 * m[-1]) ^ m[-1])
    assert m == [1, 3, 5, 15, 17, 51, 85, 255]
    pts = bf.sobol8_points(2, 0, 256)
    assert [pts[1 << j] for j in range(8)] == [mk << (8 - (j + 1)) for j, mk in enumerate(m)]


@pytest.mark.parametrize("dim", [1, 2])
def test_sobol_matches_independent_construction(oracle_mod, dim):
    for shift in (0, 1, 77, 255):
        assert list(map(int, oracle_mod.sobol8(dim, shift))) == bf.sobol8_points(dim, shift)


def test_sobol_is_a_0m2_net(oracle_mod):
    # every aligned block of 2^m points puts exactly one point in each elementary box
    # of area 2^-m (t = 0 for dimensions 1 and 2), also after a digital shift
    for shift1, shift2 in [(0, 0), (93, 200)]:
        x = oracle_mod.sobol8(1, shift1).astype(int)
        y = oracle_mod.sobol8(2, shift2).astype(int)
        for m in range(0, 9):
            for start in range(0, 256, 1 << m):
                xs, ys = x[start:start + (1 << m)], y[start:start + (1 << m)]
                for a in range(m + 1):
                    b = m - a
                    boxes = set(zip(xs >> (8 - a), ys >> (8 - b)))
                    assert len(boxes) == (1 << m), (m, start, a)


@pytest.mark.parametrize("polarity", [0, 1])
def test_cbsg_matches_bruteforce(oracle_mod, polarity):
    rng = np.random.default_rng(200 + polarity)
    for case in range(25):
        M, N, K = (int(x) for x in rng.integers(1, 4, 3))
        L_max = int(rng.choice([1, 7, 31, 64, 100, 256]))
        A = rng.integers(-127, 128, (M, K)).astype(np.int8)
        B = rng.integers(-127, 128, (N, K)).astype(np.int8)
        sA = rng.uniform(0.001, 0.05, M).astype(np.float32)
        sB = rng.uniform(0.001, 0.05, N).astype(np.float32)
        L = rng.integers(0, L_max + 1, M).astype(np.int32)
        seed = int(rng.integers(0, 2**40))
        c, o = oracle_mod.sc_gemm_cbsg(A, B, sA, sB, L, L_max, polarity, seed)
        cb, ob = bf.cbsg_gemm(A.tolist(), B.tolist(), sA.tolist(), sB.tolist(), L.tolist(),
                              polarity, seed)
        assert c.tolist() == cb, case
        for i in range(M):
            for j in range(N):
                e = ob[i][j]
                if e == 0:
                    assert o[i, j] == 0.0
                else:
                    assert abs(Fraction(o[i, j]) - e) <= abs(e) * Fraction(1, 10**14)


def _prefix_count(r, beta, n):
    return int(np.count_nonzero(np.asarray(r[:n], np.int64) < beta))


def test_cbsg_closed_form_and_full_period(oracle_mod):
    # X = C(bB, cA) + (L - cA) - C(bB, L - cA) with cA = #{l < L : rA_l < bA} and
    # C(b, n) = #{k < n : rB_k < b}; over the full period cA = bA exactly
    rng = np.random.default_rng(7)
    seed = 99
    rA = oracle_mod.sobol8(1, oracle_mod.sobol_shift(seed, 0))
    rB = oracle_mod.sobol8(2, oracle_mod.sobol_shift(seed, 1))
    A = rng.integers(-127, 128, (6, 9)).astype(np.int8)
    B = rng.integers(-127, 128, (5, 9)).astype(np.int8)
    L = np.array([0, 1, 77, 128, 200, 256], np.int32)
    c, _ = oracle_mod.sc_gemm_cbsg(A, B, np.ones(6, np.float32), np.ones(5, np.float32), L, 256, 0, seed)
    for i in range(6):
        for j in range(5):
            x = 0
            for d in range(9):
                ba, bb = bf.beta_bipolar(int(A[i, d])), bf.beta_bipolar(int(B[j, d]))
                ca = _prefix_count(rA, ba, L[i])
                if L[i] == 256:
                    assert ca == ba
                x += _prefix_count(rB, bb, ca) + (L[i] - ca) - _prefix_count(rB, bb, L[i] - ca)
            assert c[i, j] == x
    cu, _ = oracle_mod.sc_gemm_cbsg(A, B, np.ones(6, np.float32), np.ones(5, np.float32), L, 256, 1, seed)
    for i in range(6):
        for j in range(5):
            s = 0
            for d in range(9):
                ba, bb = bf.beta_unipolar(int(A[i, d])), bf.beta_unipolar(int(B[j, d]))
                p = _prefix_count(rB, bb, _prefix_count(rA, ba, L[i]))
                s += p if (A[i, d] < 0) == (B[j, d] < 0) else -p
            assert cu[i, j] == s


def test_cbsg_error_falls_like_one_over_L(oracle_mod):
    # low-discrepancy streams with conditional generation: the error of one decoded
    # product falls like 1/L (the tolerance table of Sec. 3.2 has alpha * L nearly
    # constant), against 1/sqrt(L) for independent pseudo-random streams
    rng = np.random.default_rng(8)
    A = rng.integers(-127, 128, (1, 300)).astype(np.int8)
    B = rng.integers(-127, 128, (1, 300)).astype(np.int8)
    uA = 2.0 * np.array([bf.beta_bipolar(int(q)) for q in A[0]]) / 256 - 1
    uB = 2.0 * np.array([bf.beta_bipolar(int(q)) for q in B[0]]) / 256 - 1
    rms = {}
    for Lv in (16, 32, 64, 128, 256):
        errs = []
        for seed in range(12):
            for d in range(0, 300, 5):
                c, _ = oracle_mod.sc_gemm_cbsg(A[:, d:d + 1], B[:, d:d + 1], np.ones(1, np.float32),
                                               np.ones(1, np.float32), np.array([Lv], np.int32), 256, 0,
                                               seed)
                errs.append((2.0 * c[0, 0] - Lv) / Lv - uA[d] * uB[d])
        rms[Lv] = float(np.sqrt(np.mean(np.square(errs))))
    assert rms[16] / rms[256] > 6.0            # 1/L would give 16, 1/sqrt(L) gives 4
    for Lv in (16, 32, 64, 128, 256):
        assert 0.2 < rms[Lv] * Lv < 5.0


def test_cbsg_scc_is_small(oracle_mod):
    # conditional generation drives the stochastic cross-correlation of Eq. (3) to ~0
    seed = 5
    rA = oracle_mod.sobol8(1, oracle_mod.sobol_shift(seed, 0)).astype(int)
    rB = oracle_mod.sobol8(2, oracle_mod.sobol_shift(seed, 1)).astype(int)
    from test_oracle_gemm import _scc
    vals = []
    for ba in range(16, 256, 24):
        for bb in range(16, 256, 24):
            za = (rA < ba).astype(np.int64)
            zb = np.zeros(256, np.int64)
            k1 = k0 = 0
            for l in range(256):
                if za[l]:
                    zb[l] = rB[k1] < bb
                    k1 += 1
                else:
                    zb[l] = rB[k0] < bb
                    k0 += 1
            vals.append(abs(_scc(za, zb)))
    assert np.mean(vals) < 0.05


def test_zero_a_is_an_exact_zero_of_the_product(oracle_mod):
    """Eq. (6): gating makes B's bits on A's 1-cycles and on its 0-cycles both follow B's own
    sequence, so the product is bias-free at finite L (App. A.1: ad - bc = 0).  For A = 0
    (boundary 128) and L = 2^m, the first L points of dimension 1 put exactly L/2 of A's bits
    at 1, B's generator then runs the same prefix of L/2 draws on both branches, and the XNOR
    count is L/2 for every B value and seed: the decode is exactly 0.  Streams from the same
    two Sobol dimensions without gating miss this for about half of the (B, L, seed) cases,
    so the property pins the gating itself."""
    B = np.arange(-127, 128, dtype=np.int8).reshape(-1, 1)
    A = np.zeros((1, 1), np.int8)
    ungated_misses = 0
    for seed in range(6):
        rA = oracle_mod.sobol8(1, oracle_mod.sobol_shift(seed, 0))
        rB = oracle_mod.sobol8(2, oracle_mod.sobol_shift(seed, 1))
        for m in range(1, 9):
            L = 2 ** m
            c, o = oracle_mod.sc_gemm_cbsg(A, B, np.ones(1, np.float32), np.ones(255, np.float32),
                                           np.array([L], np.int32), 256, 0, seed)
            assert np.all(c == L // 2), (seed, L)
            assert np.all(o == 0.0)
            for q in range(-127, 128):
                zA = rA[:L] < oracle_mod.beta_bipolar(0)
                zB = rB[:L] < oracle_mod.beta_bipolar(q)
                ungated_misses += int((zA == zB).sum()) != L // 2
    assert ungated_misses > 1000
