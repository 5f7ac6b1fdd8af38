"""The oracle still reproduces the frozen fixtures under tests/golden (CPU only).

The fixtures were written by tests/golden/make_golden.py from the oracle alone; a
failure here means the oracle's arithmetic changed, which must be justified by the
paper (Sec. 3.1 comparator and Eq. (1), Sec. 4.2 boundaries, Sec. A.1 LFSR).
"""
import hashlib
import os

import numpy as np

import sc_bruteforce as bf

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_golden_draws(oracle_mod):
    for seed, op, st, *r in _rows("lfsr_draws.txt"):
        seed, op = int(seed), int(op)
        assert oracle_mod.seed_state(seed, op) == int(st, 16)
        assert list(map(int, oracle_mod.comparator_sequence(seed, op, 32))) == list(map(int, r))
        assert bf.draws(seed, op, 32) == list(map(int, r))


def test_golden_beta_tables(oracle_mod):
    for q, bb, bu in _rows("beta_tables.txt"):
        assert oracle_mod.beta_bipolar(int(q)) == int(bb)
        assert oracle_mod.beta_unipolar(int(q)) == int(bu)


def test_golden_counts_64x256x64(oracle_mod):
    import workloads
    g = workloads.bipolar_64x256x64().gemms[0]
    c, _ = oracle_mod.sc_gemm(g.A[0], g.B[0], g.sA[0], g.sB[0], g.L[0], g.L_max, g.polarity, g.seed)
    with open(os.path.join(GOLD, "bipolar_64x256x64_counts.txt")) as f:
        lines = f.read().splitlines()
    sha = lines[1].split()[-1]
    gold = np.array([[int(x) for x in ln.split()] for ln in lines[2:]], np.int32)
    assert np.array_equal(c, gold)
    assert hashlib.sha256(c.astype("<i4").tobytes()).hexdigest() == sha
