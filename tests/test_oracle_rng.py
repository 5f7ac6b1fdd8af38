"""Pins of the oracle's comparator sequence and boundary maps (CPU only).

Each check compares the oracle with something other than itself: published
SplitMix64 outputs, polynomial algebra over GF(2), a pure-Python register, closed
forms of the boundary maps, and distributional properties.
"""
import numpy as np
import pytest

import gf2poly
import sc_bruteforce as bf

pytestmark = pytest.mark.filterwarnings("ignore")


def test_splitmix64_published_outputs(oracle_mod):
    # The first three outputs of SplitMix64 started from state 0 (Steele, Lea and
    # Flood 2014; the generator adds the golden-gamma before mixing).
    gamma = 0x9E3779B97F4A7C15
    assert oracle_mod.splitmix64(0) == 0xE220A8397B1DCDAF
    assert oracle_mod.splitmix64(gamma) == 0x6E789E6AA1B965F4
    assert oracle_mod.splitmix64((2 * gamma) & (2**64 - 1)) == 0x06C45D188009454F


def test_seed_states_match_bruteforce_and_differ_per_operand(oracle_mod):
    for seed in range(6):
        a, b = oracle_mod.seed_state(seed, 0), oracle_mod.seed_state(seed, 1)
        assert a == bf.seed_state(seed, 0) and b == bf.seed_state(seed, 1)
        assert a != b and a != 0 and b != 0


def test_order_of_two_pow32_minus_one_factorisation():
    prod = 1
    for f in gf2poly.ORDER_PRIME_FACTORS:
        prod *= f
    assert prod == gf2poly.ORDER


def test_feedback_polynomial_is_primitive():
    # x has order exactly 2^32-1 in GF(2)[x]/p  <=>  p is primitive  <=>  the
    # register visits every non-zero state before repeating.
    assert gf2poly.ppow(2, gf2poly.ORDER) == 1
    for f in gf2poly.ORDER_PRIME_FACTORS:
        assert gf2poly.ppow(2, gf2poly.ORDER // f) != 1


def test_register_step_is_multiplication_by_x_inverse(oracle_mod):
    xinv = gf2poly.x_inverse()
    assert xinv == 0x80200003       # x * (x^31 + x^21 + x + 1) = p(x) + 1
    rng = np.random.default_rng(11)
    for _ in range(20):
        s0 = int(rng.integers(1, 2**32))
        states = oracle_mod.lfsr_states(s0, 200)
        acc = s0
        for n in range(200):
            acc = gf2poly.pmul(acc, xinv)
            assert int(states[n]) == acc


def test_draws_follow_polynomial_definition(oracle_mod):
    # Output bit of step k is the constant coefficient of S_0 * x^{-k}; a draw packs
    # 8 consecutive output bits, the first one most significant.
    xinv = gf2poly.x_inverse()
    for seed, op in [(0, 0), (0, 1), (3, 1), (123456789, 0)]:
        s0 = oracle_mod.seed_state(seed, op)
        r = oracle_mod.comparator_sequence(seed, op, 40)
        acc = s0
        bits = []
        for _ in range(8 * 40):
            bits.append(acc & 1)
            acc = gf2poly.pmul(acc, xinv)
        expect = [int("".join(map(str, bits[8 * l:8 * l + 8])), 2) for l in range(40)]
        assert list(map(int, r)) == expect
        assert list(map(int, r)) == bf.draws(seed, op, 40)


def test_jump_ahead_identity(oracle_mod):
    # state after n steps from S_0 equals S_0 * J_n with J_n the state after n steps
    # from the constant polynomial 1: the parallel generator of a later kernel can
    # rely on this.
    rng = np.random.default_rng(5)
    for _ in range(10):
        s0 = int(rng.integers(1, 2**32))
        n = int(rng.integers(1, 5000))
        sn = int(oracle_mod.lfsr_states(s0, n)[-1])
        jn = int(oracle_mod.lfsr_states(1, n)[-1])
        assert sn == gf2poly.pmul(s0, jn)


def test_draws_are_uniform_bytes(oracle_mod):
    r = oracle_mod.comparator_sequence(7, 0, 1 << 16).astype(np.int64)
    hist = np.bincount(r, minlength=256)
    expect = len(r) / 256.0
    chi2 = float(((hist - expect) ** 2 / expect).sum())
    # 255 degrees of freedom: mean 255, sd ~22.6; 6 sd bound
    assert 100 < chi2 < 255 + 6 * 22.6
    # consecutive draws share no bits: lag-1 correlation near 0
    x = r - r.mean()
    rho = float((x[1:] * x[:-1]).mean() / x.var())
    assert abs(rho) < 0.02


def test_beta_bipolar_closed_form(oracle_mod):
    b = np.array([oracle_mod.beta_bipolar(q) for q in range(-127, 128)])
    assert b[0] == 0 and b[127] == 128 and b[254] == 256
    assert np.all(np.diff(b) >= 1)                       # strictly increasing
    assert np.all(b + b[::-1] == 256)                    # beta(-q) = 256 - beta(q)
    q = np.arange(-127, 128)
    # probability of a one, beta/256, against the encoding (v+1)/2 with v = q/127
    err = np.abs(b / 256.0 - (q / 127.0 + 1) / 2)
    assert err.max() <= 1 / 512 + 1e-12
    assert list(b) == [bf.beta_bipolar(int(x)) for x in q]


def test_beta_unipolar_closed_form(oracle_mod):
    q = np.arange(-127, 128)
    b = np.array([oracle_mod.beta_unipolar(int(x)) for x in q])
    assert oracle_mod.beta_unipolar(0) == 0
    assert oracle_mod.beta_unipolar(127) == 256 and oracle_mod.beta_unipolar(-127) == 256
    assert np.all(b == b[::-1])                          # depends on |q| only
    mag = b[127:]
    assert np.all(np.diff(mag) >= 2)                     # 256/127 > 2 per level
    err = np.abs(mag / 256.0 - np.arange(128) / 127.0)
    assert err.max() <= 1 / 512 + 1e-12
    assert list(b) == [bf.beta_unipolar(int(x)) for x in q]
