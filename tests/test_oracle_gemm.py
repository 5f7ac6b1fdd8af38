"""Pins of the oracle's SC GEMM (CPU only).

The oracle is checked against: an independent pure-Python brute force; closed
forms (constant operands turn a count into a count of draws below a threshold);
an independent pair-count formulation; invariants (count range, nesting, K-split
additivity, permutation equivariance, prefix consistency, one-bit flips); the
exact rational decode of Eq. (1); and statistical properties that the paper
states (unbiasedness, per-pair variance, convergence in L, zero mean SCC).
"""
from fractions import Fraction

import numpy as np
import pytest

import sc_bruteforce as bf

BIP, UNI = 0, 1


def _rand_case(rng, M, N, K, L_max, L_lo=0):
    A = rng.integers(-127, 128, (M, K)).astype(np.int8)
    B = rng.integers(-127, 128, (N, K)).astype(np.int8)
    sA = rng.uniform(0.001, 0.05, M).astype(np.float32)
    sB = rng.uniform(0.001, 0.05, N).astype(np.float32)
    L = rng.integers(L_lo, L_max + 1, M).astype(np.int32)
    return A, B, sA, sB, L


@pytest.mark.parametrize("polarity", [BIP, UNI])
def test_matches_pure_python_bruteforce(oracle_mod, polarity):
    rng = np.random.default_rng(100 + polarity)
    for case in range(40):
        M, N, K = (int(x) for x in rng.integers(1, 4, 3))
        L_max = int(rng.choice([0, 1, 5, 31, 32, 33, 64]))
        A, B, sA, sB, L = _rand_case(rng, M, N, K, L_max)
        seed = int(rng.integers(0, 2**40))
        c, o = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max, polarity, seed)
        cb, ob = bf.sc_gemm(A.tolist(), B.tolist(), sA.tolist(), sB.tolist(), L.tolist(),
                            polarity, seed)
        assert c.tolist() == cb, (case, M, N, K, L_max)
        for i in range(M):
            for j in range(N):
                exact = ob[i][j]
                if exact == 0:
                    assert o[i, j] == 0.0
                else:
                    assert abs(Fraction(o[i, j]) - exact) <= abs(exact) * Fraction(1, 10**14)


@pytest.mark.parametrize("polarity", [BIP, UNI])
def test_decode_matches_exact_rational_decode(oracle_mod, polarity):
    # oracle.decode applied to the brute force's counts against the brute force's exact
    # rational Eq. (1), and equal to the decode inside the oracle's GEMM
    rng = np.random.default_rng(140 + polarity)
    for case in range(30):
        M, N, K = (int(x) for x in rng.integers(1, 4, 3))
        L_max = int(rng.choice([0, 1, 5, 32, 33, 64]))
        A, B, sA, sB, L = _rand_case(rng, M, N, K, L_max)
        seed = int(rng.integers(0, 2**40))
        cb, ob = bf.sc_gemm(A.tolist(), B.tolist(), sA.tolist(), sB.tolist(), L.tolist(),
                            polarity, seed)
        o = oracle_mod.decode(np.array(cb, np.int32).reshape(M, N), sA, sB, L, K, polarity)
        for i in range(M):
            for j in range(N):
                exact = ob[i][j]
                if exact == 0:
                    assert o[i, j] == 0.0
                else:
                    assert abs(Fraction(o[i, j]) - exact) <= abs(exact) * Fraction(1, 10**14)
        c, og = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max, polarity, seed)
        assert np.array_equal(o, og)


def test_decode_closed_forms(oracle_mod):
    # counts at their extremes decode to +-(scale product) K; the midpoint count to 0;
    # one count step moves the bipolar decode by 2/L and the unipolar one by 1/L of the scale
    sA = np.array([0.5, 0.25, 1.0], np.float32)
    sB = np.array([2.0, 4.0], np.float32)
    L = np.array([64, 32, 0], np.int32)
    K = 10
    X = np.array([[640, 0], [160, 161], [5, 5]], np.int32)
    o = oracle_mod.decode(X, sA, sB, L, K, BIP)
    assert o[0, 0] == 0.5 * 2.0 * 16129 * K and o[0, 1] == -0.5 * 4.0 * 16129 * K
    assert o[1, 0] == 0.0 and o[1, 1] == 0.25 * 4.0 * 16129 * (2.0 / 32)
    assert np.all(o[2] == 0.0)
    S = np.array([[64, -64], [1, -1], [3, 3]], np.int32)
    u = oracle_mod.decode(S, sA, sB, L, K, UNI)
    assert u[0, 0] == 0.5 * 2.0 * 16129 and u[0, 1] == -0.5 * 4.0 * 16129
    assert u[1, 0] == 0.25 * 2.0 * 16129 / 32 and np.all(u[2] == 0.0)


def test_count_range_and_zero_length(oracle_mod):
    rng = np.random.default_rng(1)
    A, B, sA, sB, L = _rand_case(rng, 9, 7, 37, 70)
    L[:3] = 0
    for pol in (BIP, UNI):
        c, o = oracle_mod.sc_gemm(A, B, sA, sB, L, 70, pol, 9)
        KL = 37 * L[:, None]
        if pol == BIP:
            assert np.all((c >= 0) & (c <= KL))
        else:
            assert np.all(np.abs(c) <= KL)
        assert np.all(c[:3] == 0) and np.all(o[:3] == 0.0)


def _count_below(r, beta, L):
    """#{l < L : r_l < beta} for vectors beta (independent of the oracle's loops)."""
    srt = np.sort(r[:L].astype(np.int64))
    return np.searchsorted(srt, np.asarray(beta, np.int64), side="left")


def test_constant_operand_closed_forms(oracle_mod):
    # bipolar: B = +127 has beta = 256, all-ones streams, so XNOR(a, 1) = a and
    # X_ij = sum_d #{l < L_i : rA_l < beta(A_id)}; B = -127 is all zeros and counts
    # the complement.  Unipolar: |B| = 127 is all ones, so S_ij sums the signed
    # magnitudes of A's streams, i.e. the AND multiplier returns the other operand.
    rng = np.random.default_rng(2)
    M, K, L_max, seed = 6, 50, 200, 77
    A = rng.integers(-127, 128, (M, K)).astype(np.int8)
    L = rng.integers(0, L_max + 1, M).astype(np.int32)
    sA = np.ones(M, np.float32)
    rA = oracle_mod.comparator_sequence(seed, 0, L_max)
    beta_b = np.array([[bf.beta_bipolar(int(q)) for q in row] for row in A])
    beta_u = np.array([[bf.beta_unipolar(int(q)) for q in row] for row in A])
    Bp = np.full((2, K), 127, np.int8)
    Bp[1] = -127
    c, _ = oracle_mod.sc_gemm(A, Bp, sA, np.ones(2, np.float32), L, L_max, BIP, seed)
    for i in range(M):
        ones = _count_below(rA, beta_b[i], L[i]).sum()
        assert c[i, 0] == ones
        assert c[i, 1] == K * L[i] - ones
    c, _ = oracle_mod.sc_gemm(A, Bp, sA, np.ones(2, np.float32), L, L_max, UNI, seed)
    sign = np.where(A < 0, -1, 1)
    for i in range(M):
        signed = (sign[i] * _count_below(rA, beta_u[i], L[i])).sum()
        assert c[i, 0] == signed and c[i, 1] == -signed


def test_pair_count_formulation(oracle_mod):
    # Under a shared sequence per operand a pair's count depends only on the two
    # boundaries and L: P_L[ba, bb] = #{l < L : (rA_l < ba) == (rB_l < bb)}.
    rng = np.random.default_rng(3)
    M, N, K, L_max, seed = 5, 6, 40, 96, 1234
    A, B, sA, sB, L = _rand_case(rng, M, N, K, L_max)
    c, _ = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max, BIP, seed)
    rA = oracle_mod.comparator_sequence(seed, 0, L_max).astype(np.int64)
    rB = oracle_mod.comparator_sequence(seed, 1, L_max).astype(np.int64)
    levels = np.arange(257)
    zA = (rA[None, :] < levels[:, None])          # [257, L_max]
    zB = (rB[None, :] < levels[:, None])
    bA = np.vectorize(bf.beta_bipolar)(A.astype(np.int64))
    bB = np.vectorize(bf.beta_bipolar)(B.astype(np.int64))
    for i in range(M):
        Li = int(L[i])
        P = (zA[:, None, :Li] == zB[None, :, :Li]).sum(axis=2)   # [257, 257]
        expect = P[bA[i][None, :], bB].sum(axis=1)                  # over d
        assert np.array_equal(c[i], expect)


@pytest.mark.parametrize("polarity", [BIP, UNI])
def test_k_split_additivity_and_permutations(oracle_mod, polarity):
    rng = np.random.default_rng(4 + polarity)
    M, N, K, L_max, seed = 7, 9, 61, 80, 42
    A, B, sA, sB, L = _rand_case(rng, M, N, K, L_max)
    c, _ = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max, polarity, seed)
    k1 = 23
    c1, _ = oracle_mod.sc_gemm(A[:, :k1], B[:, :k1], sA, sB, L, L_max, polarity, seed)
    c2, _ = oracle_mod.sc_gemm(A[:, k1:], B[:, k1:], sA, sB, L, L_max, polarity, seed)
    assert np.array_equal(c, c1 + c2)
    pr, pc, pk = rng.permutation(M), rng.permutation(N), rng.permutation(K)
    cp, _ = oracle_mod.sc_gemm(A[pr][:, pk], B[pc][:, pk], sA[pr], sB[pc], L[pr], L_max,
                               polarity, seed)
    assert np.array_equal(cp, c[pr][:, pc])


@pytest.mark.parametrize("polarity", [BIP, UNI])
def test_prefix_consistency(oracle_mod, polarity):
    # Row i under a per-row length L_i equals the same row under a uniform length
    # L_i: early termination takes a prefix of the same streams (Sec. 3.1, Sec. 4.2).
    rng = np.random.default_rng(6)
    M, N, K, L_max, seed = 6, 5, 33, 150, 5
    A, B, sA, sB, L = _rand_case(rng, M, N, K, L_max)
    c, o = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max, polarity, seed)
    for i in range(M):
        Lu = np.full(M, L[i], np.int32)
        cu, ou = oracle_mod.sc_gemm(A, B, sA, sB, Lu, L_max, polarity, seed)
        assert np.array_equal(cu[i], c[i]) and np.array_equal(ou[i], o[i])
    # a larger L_max only appends draws: results do not change
    c2, _ = oracle_mod.sc_gemm(A, B, sA, sB, L, L_max + 77, polarity, seed)
    assert np.array_equal(c, c2)


def test_streams_nested_and_extremes(oracle_mod):
    X = np.arange(-127, 128, dtype=np.int8)[None, :]
    for pol in (BIP, UNI):
        z = oracle_mod.streams(X, pol, 9, 0, 300)[0]      # [255, 300]
        beta = [bf.beta_bipolar(q) if pol == BIP else bf.beta_unipolar(q) for q in range(-127, 128)]
        order = np.argsort(beta, kind="stable")
        zs = z[order].astype(np.int64)
        assert np.all(zs[1:] >= zs[:-1])                   # monotone comparator: nested
        for q, row in zip(range(-127, 128), z):
            b = beta[q + 127]
            if b == 256:
                assert row.all()
            if b == 0:
                assert not row.any()


def test_one_bit_flip_moves_decode_by_2_over_L(oracle_mod):
    # Change one element of B by one level so that exactly one comparator bit of
    # its stream flips within L cycles; the count moves by exactly 1 and the decode
    # by exactly 2/L (bipolar) or 1/L (unipolar) times s^A s^B q_max^2.
    seed, L, K = 21, 64, 8
    rB = oracle_mod.comparator_sequence(seed, 1, L).astype(np.int64)
    rng = np.random.default_rng(8)
    A = rng.integers(-127, 128, (1, K)).astype(np.int8)
    sA = np.array([0.25], np.float32)
    sB = np.array([0.5, 0.5], np.float32)
    for pol in (BIP, UNI):
        betaf = bf.beta_bipolar if pol == BIP else bf.beta_unipolar
        found = 0
        for q in range(1, 127):
            b0, b1 = betaf(q), betaf(q + 1)
            flips = int(((rB[:L] >= b0) & (rB[:L] < b1)).sum())
            if flips != 1:
                continue
            B = np.tile(rng.integers(-127, 128, (1, K)).astype(np.int8), (2, 1))
            B[0, 3], B[1, 3] = q, q + 1
            c, o = oracle_mod.sc_gemm(A, B, sA, sB, np.array([L], np.int32), L, pol, seed)
            za = oracle_mod.streams(A[:, 3:4], pol, seed, 0, L)[0, 0]
            flip_pos = np.nonzero((rB[:L] >= b0) & (rB[:L] < b1))[0][0]
            a_bit = int(za[flip_pos])
            if pol == BIP:
                step = 1 if a_bit == 1 else -1          # B's bit turns 0 -> 1
            else:
                step = a_bit * (1 if A[0, 3] >= 0 else -1)
            assert c[0, 1] - c[0, 0] == step
            unit = 0.25 * 0.5 * 127 * 127 * (2.0 if pol == BIP else 1.0) / L
            assert o[0, 1] - o[0, 0] == pytest.approx(step * unit, rel=0, abs=1e-9)
            found += 1
        assert found >= 3


def _scc(za, zb):
    """Stochastic cross-correlation, Eq. (3), from the bit-pair counts a, b, c, d."""
    L = len(za)
    a = int(np.sum(za & zb)); b = int(np.sum(za & (1 - zb)))
    c = int(np.sum((1 - za) & zb)); d = int(np.sum((1 - za) & (1 - zb)))
    num = a * d - b * c
    if num > 0:
        den = L * min(a + b, a + c) - (a + b) * (a + c)
    else:
        den = (a + b) * (a + c) - L * max(a - d, 0)
    return 0.0 if den == 0 else num / den


def test_scc_definition_extremes():
    z = np.array([1, 0, 1, 1, 0, 0, 1, 0], np.int64)
    assert _scc(z, z) == pytest.approx(1.0)
    assert _scc(z, 1 - z) == pytest.approx(-1.0)
    x = np.array([1, 1, 0, 0], np.int64); y = np.array([1, 0, 1, 0], np.int64)
    assert _scc(x, y) == 0.0                              # ad - bc = 1*1 - 1*1


def test_unbiased_over_seeds_and_variance(oracle_mod):
    # Sec. 3.1: E[C_hat] = C for independent streams and the per-pair estimator has
    # variance (1 - (uA uB)^2) / L.  Here u is the encoded value 2 beta/256 - 1.
    rng = np.random.default_rng(9)
    K, L, S = 1, 64, 1500
    A = rng.integers(-127, 128, (6, K)).astype(np.int8)
    B = rng.integers(-127, 128, (5, K)).astype(np.int8)
    ones6, ones5 = np.ones(6, np.float32), np.ones(5, np.float32)
    Ls = np.full(6, L, np.int32)
    est = np.zeros((S, 6, 5))
    sccs = []
    for s in range(S):
        c, _ = oracle_mod.sc_gemm(A, B, ones6, ones5, Ls, L, BIP, 1000 + s)
        est[s] = (2.0 * c - L) / L
        if s < 300:
            za = oracle_mod.streams(A[:1], BIP, 1000 + s, 0, L)[0, 0].astype(np.int64)
            zb = oracle_mod.streams(B[:1], BIP, 1000 + s, 1, L)[0, 0].astype(np.int64)
            sccs.append(_scc(za, zb))
    uA = 2.0 * np.vectorize(bf.beta_bipolar)(A[:, 0].astype(int)) / 256 - 1
    uB = 2.0 * np.vectorize(bf.beta_bipolar)(B[:, 0].astype(int)) / 256 - 1
    prod = uA[:, None] * uB[None, :]
    var = (1 - prod ** 2) / L
    mean = est.mean(axis=0)
    assert np.all(np.abs(mean - prod) <= 4.5 * np.sqrt(var / S) + 1e-12)
    emp = est.var(axis=0)
    assert np.all(np.abs(emp - var) <= 0.15 * var + 1e-4)
    sccs = np.array(sccs)
    assert abs(sccs.mean()) <= 4.5 * sccs.std() / np.sqrt(len(sccs))


def test_error_shrinks_like_inverse_sqrt_L(oracle_mod):
    rng = np.random.default_rng(10)
    A = rng.integers(-127, 128, (1, 400)).astype(np.int8)
    B = rng.integers(-127, 128, (1, 400)).astype(np.int8)
    uA = 2.0 * np.vectorize(bf.beta_bipolar)(A[0].astype(int)) / 256 - 1
    uB = 2.0 * np.vectorize(bf.beta_bipolar)(B[0].astype(int)) / 256 - 1
    # K = 1 pairs, one column per pair, over many independent seeds
    rms = []
    Ls = [64, 256, 1024, 4096]
    for L in Ls:
        errs = []
        for s in range(40):
            c = np.array([oracle_mod.sc_gemm(A[:, k:k + 1], B[:, k:k + 1], np.ones(1, np.float32),
                                             np.ones(1, np.float32), np.array([L], np.int32), L,
                                             BIP, 7 + s)[0][0, 0] for k in range(0, 400, 20)])
            est = (2.0 * c - L) / L
            errs.append(est - uA[::20] * uB[::20])
        errs = np.concatenate(errs)
        expect = np.sqrt(np.mean(1 - (uA[::20] * uB[::20]) ** 2) / L)
        rms.append(np.sqrt(np.mean(errs ** 2)))
        assert 0.5 * expect <= rms[-1] <= 2.0 * expect
    assert rms[0] > rms[1] > rms[2] > rms[3]
