"""GPU parity: the HIP library against the CPU oracle, through the C ABI.

Counts must agree bit for bit; decoded floats within 1e-6 relative (exact zeros on
both sides).  The 1e-6 bound follows from the decode arithmetic: the integer
numerator (2X - K L or S) is exact, then one fp32 division by L and two fp32
products with the scales, i.e. at most four roundings of 2^-24 each (< 2.4e-7).

Small cases span several 128x128 tiles with ragged tails and run the oracle on every
output; the five full-size workloads (the launch configuration the benchmark times)
are checked on sampled rows x columns, plus whole-matrix properties.
"""
import sys

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

REL_TOL = 1e-6


def _note(msg):
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_32922_amd as scg
    scg.load()
    return torch.device("cuda:0")


def _to_dev(g, dev):
    import torch
    return (torch.from_numpy(np.ascontiguousarray(g.A)).to(dev),
            torch.from_numpy(np.ascontiguousarray(g.sA)).to(dev),
            torch.from_numpy(np.ascontiguousarray(g.B)).to(dev),
            torch.from_numpy(np.ascontiguousarray(g.sB)).to(dev),
            torch.from_numpy(np.ascontiguousarray(g.L)).to(dev))


def _run(g, dev, check_status=True, rng=0, L_hint=0):
    import torch
    import paper_2609_32922_amd as scg
    A, sA, B, sB, L = _to_dev(g, dev)
    out, cnt = scg.gemm(A, sA, B, sB, L, L_max=g.L_max, polarity=g.polarity, seed=g.seed,
                        want_counts=True, check_status=check_status, rng=rng, L_hint=L_hint)
    torch.cuda.synchronize()
    return out.cpu().numpy(), cnt.cpu().numpy()


def _compare(g, b, rows, cols, out, cnt, oracle_mod, tag, rng=0):
    bB = 0 if g.B.shape[0] == 1 else b
    ref = oracle_mod.sc_gemm_cbsg if rng == 1 else oracle_mod.sc_gemm
    c_ref, o_ref = ref(g.A[b][rows], g.B[bB][cols], g.sA[b][rows], g.sB[bB][cols],
                       g.L[b][rows], g.L_max, g.polarity, g.seed)
    c_gpu = cnt[b][np.ix_(rows, cols)]
    o_gpu = out[b][np.ix_(rows, cols)].astype(np.float64)
    bad = np.argwhere(c_gpu != c_ref)
    assert bad.size == 0, "%s: %d count mismatches, first at %s: gpu %d oracle %d" % (
        tag, len(bad), bad[0], c_gpu[tuple(bad[0])], c_ref[tuple(bad[0])])
    zero = o_ref == 0.0
    assert np.all(o_gpu[zero] == 0.0), tag + ": expected exact zeros"
    rel = np.abs(o_gpu[~zero] - o_ref[~zero]) / np.abs(o_ref[~zero])
    assert rel.size == 0 or rel.max() <= REL_TOL, "%s: max rel err %.3g" % (tag, rel.max())


def test_comparator_sequence_matches_oracle(dev, oracle_mod):
    import paper_2609_32922_amd as scg
    for seed in (0, 1, 2, 3, 4, 2**63 + 12345):
        for op in (0, 1):
            _note("comparator seed=%d op=%d" % (seed, op))
            r = scg.comparator_sequence(seed, op, 4096).cpu().numpy()
            assert np.array_equal(r, oracle_mod.comparator_sequence(seed, op, 4096))


def test_bipolar_64x256x64_full(dev, oracle_mod):
    g = W.bipolar_64x256x64().gemms[0]
    _note("bipolar_64x256x64 full")
    out, cnt = _run(g, dev)
    _compare(g, 0, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod, "64x256x64")


FUZZ = [
    # batch, M, N, K, L_max, L_lo, polarity, broadcast_B, seed
    (1, 1, 1, 1, 1, 0, 0, False, 3),
    (1, 129, 130, 33, 70, 0, 0, False, 5),
    (1, 300, 257, 100, 257, 0, 0, False, 7),
    (1, 257, 129, 64, 64, 64, 0, False, 9),
    (2, 140, 131, 96, 40, 0, 0, False, 11),
    (3, 70, 200, 31, 100, 1, 0, True, 13),
    (1, 129, 130, 33, 70, 0, 1, False, 15),
    (1, 300, 257, 100, 193, 0, 1, False, 17),
    (2, 140, 131, 65, 48, 0, 1, True, 19),
    (1, 64, 64, 1000, 24, 0, 1, False, 21),
    (1, 200, 150, 7, 512, 400, 0, False, 23),
    # N <= 128: the MFMA engine builds its fp4 fragments from the int8 rows (unaligned rows,
    # broadcast B, a split k-range with few tiles, the octet table changing every stage)
    (1, 300, 100, 33, 70, 0, 0, False, 25),
    (2, 257, 128, 65, 300, 10, 1, True, 27),
    (3, 70, 64, 130, 64, 0, 0, False, 29),
    (1, 140, 1, 5, 4096, 0, 0, False, 31),
    (2, 129, 127, 12, 200, 0, 1, False, 33),
]


@pytest.mark.parametrize("case", FUZZ, ids=[str(c) for c in FUZZ])
def test_fuzz_full_compare(dev, oracle_mod, case):
    batch, M, N, K, L_max, L_lo, pol, bcast, seed = case
    rng = np.random.default_rng(seed)
    g = W.random_gemm(rng, batch, M, N, K, L_max, pol, seed, L_lo=L_lo, broadcast_B=bcast)
    _note("fuzz %s" % (case,))
    out, cnt = _run(g, dev)
    for b in range(batch):
        _compare(g, b, np.arange(M), np.arange(N), out, cnt, oracle_mod, "fuzz%s b%d" % (case, b))


def test_zero_lengths_and_K0(dev, oracle_mod):
    rng = np.random.default_rng(31)
    g = W.random_gemm(rng, 1, 150, 140, 40, 64, 0, 31)
    g.L[0, ::3] = 0
    _note("zero lengths")
    out, cnt = _run(g, dev)
    assert np.all(cnt[0, ::3] == 0) and np.all(out[0, ::3] == 0)
    _compare(g, 0, np.arange(150), np.arange(140), out, cnt, oracle_mod, "zeroL")
    for pol in (0, 1):
        g0 = W.random_gemm(rng, 1, 10, 12, 0, 16, pol, 5)
        _note("K=0 polarity %d" % pol)
        out, cnt = _run(g0, dev)
        assert np.all(cnt == 0) and np.all(out == 0)


def test_out_of_range_lengths_set_status(dev):
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(41)
    g = W.random_gemm(rng, 1, 50, 20, 16, 32, 0, 41)
    g.L[0, 3] = 33
    g.L[0, 7] = -1
    _note("bad lengths")
    with pytest.raises(scg.ScError) as ei:
        _run(g, dev, check_status=True)
    assert ei.value.code == scg.SC_ERR_DEVICE_STATUS
    out, cnt = _run(g, dev, check_status=False)
    assert np.all(cnt[0, 3] == 0) and np.all(cnt[0, 7] == 0)
    g.L[0, 3] = 32
    g.L[0, 7] = 0
    _run(g, dev, check_status=True)          # a good call clears the status


def test_deterministic_repeat(dev):
    rng = np.random.default_rng(51)
    g = W.random_gemm(rng, 1, 260, 300, 160, 96, 0, 51)
    _note("determinism")
    o1, c1 = _run(g, dev)
    o2, c2 = _run(g, dev)
    assert np.array_equal(c1, c2) and np.array_equal(o1.view(np.uint32), o2.view(np.uint32))


@pytest.mark.parametrize("polarity", [0, 1])
def test_longest_streams(dev, oracle_mod, polarity):
    # L_max at the library's limit (4096 cycles), rows at exactly L_max and at 0, on a
    # ragged 300 x 270 shape (an odd count of 128-row tiles, so the 256-row MFMA blocks
    # take a padded pair); every output against the oracle
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(201 + polarity)
    g = W.random_gemm(rng, 1, 300, 270, 100, scg.SC_L_MAX_LIMIT, polarity, 201 + polarity)
    g.L[0, :7] = scg.SC_L_MAX_LIMIT
    g.L[0, 7:11] = 0
    _note("longest streams polarity %d" % polarity)
    out, cnt = _run(g, dev)
    _compare(g, 0, np.arange(300), np.arange(270), out, cnt, oracle_mod, "Lmax%d pol%d" % (g.L_max, polarity))


@pytest.mark.parametrize("polarity", [0, 1])
def test_split_partials_extreme(dev, oracle_mod, polarity):
    # ViT-B fc1's shape (its last 44 tiles are split along k) with constant operands, so that
    # the parts' partial sums reach their largest magnitudes (every product +1 or -1), of both
    # signs across columns.  Equal rows of equal length give equal counts, which checks every
    # row; sampled rows, most in the split tiles, go against the oracle.
    M, N, K, L = 6304, 3072, 768, 128
    rng = np.random.default_rng(301 + polarity)
    g = W.random_gemm(rng, 1, M, N, K, L, polarity, 301 + polarity, uniform_L=L)
    g.A[:] = 127
    g.B[:] = np.where(np.arange(N)[:, None] % 2 == 0, 127, -127).astype(np.int8)
    _note("split partials extreme polarity %d" % polarity)
    out, cnt = _run(g, dev)
    assert np.array_equal(cnt[0], np.broadcast_to(cnt[0][:1], cnt[0].shape))
    rows = np.union1d(_sample(M, rng, 4), [0, 5375, 5376, 5600, 5900, 6200, 6303])
    _compare(g, 0, rows, np.arange(N), out, cnt, oracle_mod, "extreme pol%d" % polarity)


@pytest.mark.parametrize("polarity", [0, 1])
def test_int16_partials_at_their_bound(dev, oracle_mod, polarity):
    # 384 tiles of 256 x 256 on 256 CUs: the last 128 run in two parts of 31 chunk steps each
    # (K = 992: 31 chunks, L = 64: 2 cycle groups), the most whose partial counts are stored as
    # int16; constant operands give every part's counts the largest magnitude, 31 x 32 x 32 =
    # 31744, of both signs across columns.  (With K = 1024 the parts hold 32 steps and int32.)
    M, N, K, L = 6144, 4096, 992, 64
    rng = np.random.default_rng(311 + polarity)
    g = W.random_gemm(rng, 1, M, N, K, L, polarity, 311 + polarity, uniform_L=L)
    g.A[:] = 127
    g.B[:] = np.where(np.arange(N)[:, None] % 2 == 0, 127, -127).astype(np.int8)
    _note("int16 partials at the bound polarity %d" % polarity)
    out, cnt = _run(g, dev)
    assert np.array_equal(cnt[0], np.broadcast_to(cnt[0][:1], cnt[0].shape))
    rows = np.union1d(_sample(M, rng, 3), [0, 4095, 4096, 5000, 6143])
    _compare(g, 0, rows, np.arange(N), out, cnt, oracle_mod, "int16 bound pol%d" % polarity)


# --------------------------------------------------------------------------
# 256 x 256 MFMA GEMM with comparator streams: fp4 fragments built from int8 chunks
# through a table per 32-cycle group.  One variant masks every A fragment with its row's
# length (some length of the call is not a multiple of 32), the other lets rows that
# have ended read the padding byte (all lengths multiples of 32).
# --------------------------------------------------------------------------
RGEN = [
    # batch, M, N, K, L_max, lengths, polarity, broadcast_B, seed
    (1, 300, 270, 100, 160, "mult32", 0, False, 61),   # rows end at group bounds, some at 0
    (2, 257, 300, 33, 96, "mult32", 1, True, 63),      # K one past a chunk, broadcast B
    (1, 520, 260, 16, 100, "uniform", 0, False, 65),   # one length inside a group; K < 32
    (1, 384, 257, 300, 64, "random", 1, False, 67),    # every length; split k-ranges
    (3, 140, 129, 64, 512, "uniform", 1, False, 69),   # 16 groups, one pair per batch entry
    (1, 600, 513, 45, 33, "random", 0, False, 71),     # one cycle past the first group
    # N <= 64: blocks of 256 rows x 64 columns, two per CU
    (2, 300, 64, 64, 256, "uniform", 0, True, 73),     # the compensator's shape class
    (3, 577, 17, 200, 130, "random", 1, False, 75),    # attention-like, ragged N
    (1, 129, 1, 5, 96, "mult32", 0, False, 77),        # one column, K < 32, rows ending at bounds
    # one length per batch entry (the scheduler keeps the row order): inside a group with
    # 64-column blocks (every fragment masked), all rows of length 0, and per-entry lengths
    (2, 400, 48, 70, 90, "uniform", 1, False, 79),
    (1, 300, 300, 40, 64, "zero", 0, False, 81),
    (3, 600, 260, 96, 160, "per_entry", 0, True, 83),
    # 64-column blocks whose last chunk of K holds few elements (the waves run only the
    # k-steps that reach them)
    (1, 700, 64, 108, 200, "random", 0, False, 85),
    (2, 333, 20, 99, 64, "random", 1, False, 87),
    # last chunk of K holding one element (K % 32 = 1, as attention-V's K = 577) and nine (the
    # k-half 1 waves then hold one of its k-steps): the chunk runs only those k-steps
    (2, 300, 48, 33, 96, "random", 0, False, 89),
    (1, 520, 40, 73, 64, "random", 1, False, 91),
]


def _rgen_gemm(case):
    batch, M, N, K, L_max, kind, pol, bcast, seed = case
    rng = np.random.default_rng(seed)
    g = W.random_gemm(rng, batch, M, N, K, L_max, pol, seed, broadcast_B=bcast)
    if kind == "mult32":
        g.L = (rng.integers(0, L_max // 32 + 1, g.L.shape) * 32).astype(np.int32)
    elif kind == "uniform":
        g.L = np.full(g.L.shape, L_max, np.int32)
    elif kind == "zero":
        g.L = np.zeros(g.L.shape, np.int32)
    elif kind == "per_entry":
        g.L = np.repeat(rng.integers(1, L_max + 1, (g.L.shape[0], 1)), g.L.shape[1], axis=1).astype(np.int32)
    return g


@pytest.mark.parametrize("case", RGEN, ids=[str(c) for c in RGEN])
def test_rgen_full_compare(dev, oracle_mod, case):
    g = _rgen_gemm(case)
    _note("int8-chunk GEMM %s" % (case,))
    out, cnt = _run(g, dev)
    for b in range(g.batch):
        _compare(g, b, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod, "rgen%s b%d" % (case, b))


# One row length and more 256 x 256 tiles than CUs with a partial last round: on a 256-CU
# device the full rounds run whole tiles and the last round's tiles run in k-range parts whose
# partial counts the split sum adds.  Last rounds of 32 tiles, of 44 (ragged M
# and N), inside a group (L = 100: masked tables) and after two full rounds (544 tiles).
LAST_ROUND = [
    # batch, M, N, K, L_max, lengths, polarity, broadcast_B, seed
    (4, 2304, 2048, 40, 64, "uniform", 0, False, 501),
    (3, 2500, 2500, 33, 96, "uniform", 1, False, 503),
    (2, 3577, 2716, 20, 100, "uniform", 0, True, 505),
    (2, 4352, 4096, 16, 32, "uniform", 1, False, 507),
]


@pytest.mark.parametrize("case", LAST_ROUND, ids=[str(c) for c in LAST_ROUND])
def test_rgen_partial_last_round(dev, oracle_mod, case):
    g = _rgen_gemm(case)
    _note("int8-chunk GEMM, one length, partial last round %s" % (case,))
    out, cnt = _run(g, dev)
    for b in range(g.batch):
        _compare(g, b, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod, "last_round%s b%d" % (case, b))


# With an expected mean length (L_hint) below L_max the 256-row GEMM takes its split count
# from the scheduled lengths, and the 256 x 64 blocks (N <= 64) divide their tiles by length:
# long tiles in 2, 4 or 8 parts, short ones whole.  Shapes with few tiles (so that splitting
# pays), skewed lengths spanning 1..L_max, both comparator sources and polarities.
VSPLIT = [
    # batch, M, N, K, L_max, polarity, rng, broadcast_B, seed
    (1, 1000, 520, 96, 200, 0, 0, False, 401),
    (2, 700, 300, 64, 300, 1, 0, True, 403),
    (1, 900, 40, 150, 256, 1, 0, False, 405),      # 256 x 64 blocks
    (3, 577, 33, 64, 512, 0, 0, False, 407),       # attention-like heads
    (1, 800, 400, 70, 256, 0, 1, False, 409),      # C-BSG: fp4 planes, 256-row blocks
    (1, 600, 300, 100, 256, 1, 1, False, 411),
]


@pytest.mark.parametrize("case", VSPLIT, ids=[str(c) for c in VSPLIT])
def test_length_aware_split(dev, oracle_mod, case):
    batch, M, N, K, L_max, pol, rng_kind, bcast, seed = case
    rng = np.random.default_rng(seed)
    g = W.random_gemm(rng, batch, M, N, K, L_max, pol, seed, L_lo=1, broadcast_B=bcast)
    # a skewed length distribution: few long rows, many short ones (as the policy gives)
    u = rng.random(g.L.shape)
    g.L = np.maximum(1, (L_max * u ** 4)).astype(np.int32)
    g.L[:, 0] = L_max
    hint = int(round(float(g.L.mean())))
    _note("length-aware split %s L_hint %d" % (case, hint))
    out, cnt = _run(g, dev, rng=rng_kind, L_hint=hint)
    for b in range(batch):
        _compare(g, b, np.arange(M), np.arange(N), out, cnt, oracle_mod, "vsplit%s b%d" % (case, b), rng=rng_kind)
    # the same call without the hint (every tile split alike, or none) gives the same bits
    out2, cnt2 = _run(g, dev, rng=rng_kind)
    assert np.array_equal(cnt, cnt2) and np.array_equal(out.view(np.uint32), out2.view(np.uint32))


LADDERS = [
    # lengths a row pair may hold: a ladder as the length policy gives (lengths inside a
    # cycle group read tables masked to them), exactly as many such lengths in one pair as
    # there are masked tables, and one more (the call then masks every fragment)
    ("ladder", [0, 5, 24, 48, 96, 192], 192),
    ("four", [40, 41, 42, 43], 64),
    ("five", [40, 41, 42, 43, 44], 64),
]


@pytest.mark.parametrize("polarity", [0, 1])
@pytest.mark.parametrize("case", LADDERS, ids=[c[0] for c in LADDERS])
def test_rgen_length_ladders(dev, oracle_mod, case, polarity):
    name, lengths, L_max = case
    rng = np.random.default_rng(91 + polarity)
    g = W.random_gemm(rng, 2, 300, 260, 40, L_max, polarity, 91 + polarity)
    g.L = rng.choice(np.array(lengths, np.int32), g.L.shape).astype(np.int32)
    _note("length ladder %s polarity %d" % (name, polarity))
    out, cnt = _run(g, dev)
    for b in range(g.batch):
        _compare(g, b, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod, "ladder %s pol%d b%d" % (name, polarity, b))


INT8_MIN_SHAPES = [
    # M, N, K, rng: int8-chunk GEMM (rows copied bytewise, then 16 bytes at a time), 128-row
    # planes GEMM (M <= 128), fragments from int8 rows (N <= 128), 256-row planes GEMM (C-BSG)
    (290, 300, 70, 0), (290, 300, 96, 0), (100, 300, 70, 0), (290, 100, 70, 0), (290, 300, 70, 1),
]


@pytest.mark.parametrize("polarity", [0, 1])
@pytest.mark.parametrize("shape", INT8_MIN_SHAPES, ids=[str(x) for x in INT8_MIN_SHAPES])
def test_int8_min(dev, oracle_mod, shape, polarity):
    # -128 lies outside the documented [-127, 127] but has the comparator boundaries of
    # -127 in both polarities (a unipolar magnitude boundary past 256: a one on every
    # cycle); every path must match the oracle on it, rows that end early included
    M, N, K, rng_kind = shape
    seed = 81 + 2 * polarity + rng_kind
    rng = np.random.default_rng(seed)
    g = W.random_gemm(rng, 1, M, N, K, 80, polarity, seed)
    g.A[0, ::5, ::3] = -128
    g.B[0, ::7, 1::4] = -128
    _note("int8 minimum %s polarity %d" % (shape, polarity))
    out, cnt = _run(g, dev, rng=rng_kind)
    _compare(g, 0, np.arange(M), np.arange(N), out, cnt, oracle_mod, "int8min %s pol%d" % (shape, polarity),
             rng=rng_kind)


# --------------------------------------------------------------------------
# full-size workloads: sampled rows x columns against the oracle
# --------------------------------------------------------------------------
def _sample(n, rng, k):
    base = [0, 1, n - 1, n - 2]
    base += list(range(max(0, (n // 128) * 128 - 2), min(n, (n // 128) * 128 + 2)))
    extra = rng.choice(n, size=min(k, n), replace=False).tolist()
    return np.array(sorted(set(i for i in base + extra if 0 <= i < n)), dtype=np.int64)


def _check_workload(w, dev, oracle_mod, nrows=40, ncols=96, batches=None, seq=0):
    rng = np.random.default_rng(7)
    for g in w.gemms:
        _note("%s/%s full size %s rng %d" % (w.name, g.name, g.A.shape, seq))
        out, cnt = _run(g, dev, rng=seq)
        KL = g.K * g.L.astype(np.int64)
        if g.polarity == 0:
            assert np.all(cnt >= 0) and np.all(cnt <= KL[:, :, None])
        else:
            assert np.all(np.abs(cnt) <= KL[:, :, None])
        bs = range(g.batch) if batches is None else batches
        for b in bs:
            rows = _sample(g.M, rng, nrows)
            cols = _sample(g.N, rng, ncols)
            _compare(g, b, rows, cols, out, cnt, oracle_mod, "%s/%s b%d" % (w.name, g.name, b),
                     rng=seq)


# The scheduler keeps up to 8192 lengths per batch entry in registers and loops over longer
# entries; both paths sort, validate and give the tile lengths.
SCHED_LONG = [(8192, 64, 1), (8193, 64, 0), (12000, 300, 1)]


@pytest.mark.parametrize("case", SCHED_LONG, ids=[str(c) for c in SCHED_LONG])
def test_schedule_long_batch_entries(dev, oracle_mod, case):
    import paper_2609_32922_amd as scg
    M, N, pol = case
    rng = np.random.default_rng(M + N)
    g = W.random_gemm(rng, 2, M, N, 40, 96, pol, 61)
    _note("long batch entries %s" % (case,))
    out, cnt = _run(g, dev)
    for b in range(2):
        rows = np.union1d(_sample(M, rng, 60), [r for r in (8190, 8191, 8192, 8193) if r < M])
        _compare(g, b, rows, np.arange(N), out, cnt, oracle_mod, "long M %d b%d" % (M, b))
    # an out-of-range length past the first 8192 rows is flagged and its row counts nothing
    g.L[1, M - 1] = 97
    with pytest.raises(scg.ScError) as ei:
        _run(g, dev, check_status=True)
    assert ei.value.code == scg.SC_ERR_DEVICE_STATUS
    out, cnt = _run(g, dev, check_status=False)
    assert np.all(cnt[1, M - 1] == 0)


def test_workload_vitb16_fc1_L128(dev, oracle_mod):
    _check_workload(W.vitb16_fc1_L128(), dev, oracle_mod)


def test_workload_vitb16_fc1_mp64(dev, oracle_mod):
    _check_workload(W.vitb16_fc1_mp64(), dev, oracle_mod)


def test_workload_ditxl2_proj_mlp_group96(dev, oracle_mod):
    _check_workload(W.ditxl2_proj_mlp_group96(), dev, oracle_mod)


def test_workload_vitl14_336_qk_mlp(dev, oracle_mod):
    _check_workload(W.vitl14_336_qk_mlp(), dev, oracle_mod, nrows=24, ncols=64,
                    batches=None)


def test_workload_vitl14_compensator_L256(dev, oracle_mod):
    _check_workload(W.vitl14_compensator_L256(), dev, oracle_mod, nrows=24, ncols=64)


def test_workload_vitl14_336_attn_av(dev, oracle_mod):
    _check_workload(W.vitl14_336_attn_av(), dev, oracle_mod, nrows=16, ncols=64, batches=range(0, 128, 9))


def test_strided_interleaved_heads(dev, oracle_mod):
    """Per-head GEMMs read straight out of one token matrix (lda = 1024, strideA = 64)
    and write their outputs side by side into one output matrix (ldo = 1024,
    strideO = 64): the layout of a per-head compensator on the block input."""
    import torch
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(61)
    T, H, dh = 300, 16, 64
    x = rng.integers(-127, 128, (T, H * dh)).astype(np.int8)
    sx = rng.uniform(0.01, 0.1, (H, T)).astype(np.float32)
    Wq = rng.integers(-127, 128, (H, dh, dh)).astype(np.int8)
    sw = rng.uniform(0.001, 0.01, (H, dh)).astype(np.float32)
    L = rng.integers(0, 97, (H, T)).astype(np.int32)
    d = scg.ScGemmDesc()
    d.batch, d.M, d.N, d.K = H, T, dh, dh
    d.lda, d.ldb, d.ldo = H * dh, dh, H * dh
    d.strideA, d.strideB, d.strideO = dh, dh * dh, dh
    d.strideSA, d.strideSB, d.strideL = T, dh, T
    d.L_max, d.polarity, d.rng, d.L_hint, d.seed = 96, 0, 0, 0, 77
    tx, tsx, tw, tsw, tL = (torch.from_numpy(a).to(dev) for a in (x, sx, Wq, sw, L))
    out = torch.zeros((T, H * dh), dtype=torch.float32, device=dev)
    cnt = torch.zeros((T, H * dh), dtype=torch.int32, device=dev)
    ws = scg.Workspace(scg.sc_gemm_workspace_size(d), dev)
    _note("strided interleaved heads")
    rc = scg.sc_gemm(d, tx.data_ptr(), tsx.data_ptr(), tw.data_ptr(), tsw.data_ptr(), tL.data_ptr(),
                     out.data_ptr(), cnt.data_ptr(), ws.ptr, ws.nbytes,
                     int(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    assert scg.sc_gemm_status(ws.ptr, int(torch.cuda.current_stream().cuda_stream)) == 0
    c, o = cnt.cpu().numpy(), out.cpu().numpy()
    for h in range(H):
        c_ref, o_ref = oracle_mod.sc_gemm(x[:, h * dh:(h + 1) * dh], Wq[h], sx[h], sw[h], L[h], 96, 0, 77)
        assert np.array_equal(c[:, h * dh:(h + 1) * dh], c_ref), h
        oo = o[:, h * dh:(h + 1) * dh].astype(np.float64)
        nz = o_ref != 0
        assert np.all(oo[~nz] == 0)
        assert np.max(np.abs(oo[nz] - o_ref[nz]) / np.abs(o_ref[nz])) <= 1e-6


@pytest.mark.parametrize("shift", [(0, 0), (1, 3)], ids=["aligned", "odd_bases"])
@pytest.mark.parametrize("polarity", [0, 1])
def test_rgen_strided(dev, oracle_mod, polarity, shift):
    """The int8-chunk GEMM on strided operands: A rows padded to a multiple of 16 bytes
    (16-byte chunk loads unless A's base is odd), B rows at an odd stride (loads at any byte
    alignment), a wider output row stride, two batch entries with their own strides."""
    import torch
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(71 + polarity)
    batch, M, N, K, L_max = 2, 270, 300, 96, 80
    lda, ldb, ldo = 128, 97, N + 8
    sA_, sB_, sO_ = M * lda + 32, N * ldb + 5, M * ldo + 4
    Abuf = rng.integers(-127, 128, batch * sA_).astype(np.int8)
    Bbuf = rng.integers(-127, 128, batch * sB_).astype(np.int8)
    sa = rng.uniform(0.001, 0.05, (batch, M)).astype(np.float32)
    sb = rng.uniform(0.001, 0.05, (batch, N)).astype(np.float32)
    L = rng.integers(0, L_max + 1, (batch, M)).astype(np.int32)
    L[0, :] = (L[0, :] // 32) * 32            # entry 0: lengths at group bounds
    d = scg.ScGemmDesc()
    d.batch, d.M, d.N, d.K = batch, M, N, K
    d.lda, d.ldb, d.ldo = lda, ldb, ldo
    d.strideA, d.strideB, d.strideO = sA_, sB_, sO_
    d.strideSA, d.strideSB, d.strideL = M, N, M
    d.L_max, d.polarity, d.rng, d.L_hint, d.seed = L_max, polarity, 0, 0, 171
    tA, tB, tsa, tsb, tL = (torch.from_numpy(a).to(dev) for a in (Abuf, Bbuf, sa, sb, L))
    out = torch.zeros(batch * sO_, dtype=torch.float32, device=dev)
    cnt = torch.zeros(batch * sO_, dtype=torch.int32, device=dev)
    ws = scg.Workspace(scg.sc_gemm_workspace_size(d), dev)
    _note("int8-chunk GEMM strided polarity %d" % polarity)
    sh = int(torch.cuda.current_stream().cuda_stream)
    oa, ob = shift                              # byte offsets of A's and B's bases
    rc = scg.sc_gemm(d, tA.data_ptr() + oa, tsa.data_ptr(), tB.data_ptr() + ob, tsb.data_ptr(), tL.data_ptr(),
                     out.data_ptr(), cnt.data_ptr(), ws.ptr, ws.nbytes, sh)
    assert rc == 0 and scg.sc_gemm_status(ws.ptr, sh) == 0
    c, o = cnt.cpu().numpy(), out.cpu().numpy()
    for b in range(batch):
        A = np.stack([Abuf[oa + b * sA_ + i * lda: oa + b * sA_ + i * lda + K] for i in range(M)])
        B = np.stack([Bbuf[ob + b * sB_ + j * ldb: ob + b * sB_ + j * ldb + K] for j in range(N)])
        c_ref, o_ref = oracle_mod.sc_gemm(A, B, sa[b], sb[b], L[b], L_max, polarity, 171)
        cg = np.stack([c[b * sO_ + i * ldo: b * sO_ + i * ldo + N] for i in range(M)])
        og = np.stack([o[b * sO_ + i * ldo: b * sO_ + i * ldo + N] for i in range(M)]).astype(np.float64)
        assert np.array_equal(cg, c_ref), b
        nz = o_ref != 0
        assert np.all(og[~nz] == 0)
        assert np.max(np.abs(og[nz] - o_ref[nz]) / np.abs(o_ref[nz])) <= 1e-6
        # the padding between rows and entries is left untouched
        assert np.all(c[b * sO_ + M * ldo - 8: b * sO_ + M * ldo] == 0) or ldo == N


# --------------------------------------------------------------------------
# Sobol-8 sequences with conditional generation of B's stream (C-BSG)
# --------------------------------------------------------------------------
def test_sobol_sequence_matches_oracle(dev, oracle_mod):
    import paper_2609_32922_amd as scg
    for seed in (0, 1, 5, 2**64 - 1):
        for op in (0, 1):
            _note("sobol seed=%d op=%d" % (seed, op))
            r = scg.comparator_sequence(seed, op, 256, rng=scg.SC_RNG_SOBOL8_CBSG).cpu().numpy()
            ref = oracle_mod.sobol8(op + 1, oracle_mod.sobol_shift(seed, op), 256)
            assert np.array_equal(r, ref)
            # one full period visits every 8-bit value once
            assert np.array_equal(np.sort(r), np.arange(256))


CBSG_FUZZ = [
    # batch, M, N, K, L_max, L_lo, polarity, broadcast_B, seed
    (1, 1, 1, 1, 1, 0, 0, False, 101),
    (1, 129, 130, 33, 70, 0, 0, False, 103),
    (1, 300, 257, 100, 256, 0, 0, False, 105),
    (1, 257, 129, 64, 64, 64, 0, False, 107),
    (2, 140, 131, 96, 40, 0, 0, False, 109),
    (3, 70, 200, 31, 100, 1, 0, True, 111),
    (1, 129, 130, 33, 70, 0, 1, False, 113),
    (1, 300, 257, 100, 193, 0, 1, False, 115),
    (2, 140, 131, 65, 48, 0, 1, True, 117),
    (1, 64, 64, 1000, 24, 0, 1, False, 119),
    (1, 200, 150, 7, 256, 200, 0, False, 121),
]


@pytest.mark.parametrize("case", CBSG_FUZZ, ids=[str(c) for c in CBSG_FUZZ])
def test_cbsg_fuzz_full_compare(dev, oracle_mod, case):
    batch, M, N, K, L_max, L_lo, pol, bcast, seed = case
    rng = np.random.default_rng(seed)
    g = W.random_gemm(rng, batch, M, N, K, L_max, pol, seed, L_lo=L_lo, broadcast_B=bcast)
    _note("cbsg fuzz %s" % (case,))
    out, cnt = _run(g, dev, rng=1)
    for b in range(batch):
        _compare(g, b, np.arange(M), np.arange(N), out, cnt, oracle_mod,
                 "cbsg%s b%d" % (case, b), rng=1)


def test_cbsg_extreme_values(dev, oracle_mod):
    """Saturated and zero operands: c = 0, c = L and c = L - c hit every branch of the
    interval planes (empty interval, full interval, sign flips)."""
    rng = np.random.default_rng(131)
    for pol in (0, 1):
        g = W.random_gemm(rng, 1, 140, 136, 70, 96, pol, 131 + pol)
        vals = np.array([-127, -126, -1, 0, 1, 126, 127], np.int8)
        g.A[0] = rng.choice(vals, g.A[0].shape)
        g.B[0] = rng.choice(vals, g.B[0].shape)
        _note("cbsg extremes polarity %d" % pol)
        out, cnt = _run(g, dev, rng=1)
        _compare(g, 0, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod,
                 "cbsg extremes %d" % pol, rng=1)


def test_cbsg_zero_lengths_and_K0(dev, oracle_mod):
    rng = np.random.default_rng(141)
    g = W.random_gemm(rng, 1, 150, 140, 40, 64, 0, 141)
    g.L[0, ::3] = 0
    _note("cbsg zero lengths")
    out, cnt = _run(g, dev, rng=1)
    assert np.all(cnt[0, ::3] == 0) and np.all(out[0, ::3] == 0)
    _compare(g, 0, np.arange(150), np.arange(140), out, cnt, oracle_mod, "cbsg zeroL", rng=1)
    for pol in (0, 1):
        g0 = W.random_gemm(rng, 1, 10, 12, 0, 16, pol, 5)
        _note("cbsg K=0 polarity %d" % pol)
        out, cnt = _run(g0, dev, rng=1)
        assert np.all(cnt == 0) and np.all(out == 0)


def test_cbsg_bad_lengths_set_status(dev):
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(151)
    g = W.random_gemm(rng, 1, 50, 20, 16, 32, 0, 151)
    g.L[0, 3] = 33
    _note("cbsg bad lengths")
    with pytest.raises(scg.ScError) as ei:
        _run(g, dev, check_status=True, rng=1)
    assert ei.value.code == scg.SC_ERR_DEVICE_STATUS


def test_cbsg_workload_vitb16_fc1_L128(dev, oracle_mod):
    _check_workload(W.vitb16_fc1_L128(), dev, oracle_mod, nrows=24, ncols=64, seq=1)


def test_cbsg_workload_vitb16_fc1_mp64(dev, oracle_mod):
    _check_workload(W.vitb16_fc1_mp64(), dev, oracle_mod, nrows=24, ncols=64, seq=1)


def test_cbsg_workload_ditxl2_proj_mlp_group96(dev, oracle_mod):
    _check_workload(W.ditxl2_proj_mlp_group96(), dev, oracle_mod, nrows=16, ncols=48, seq=1)


# --------------------------------------------------------------------------
# exactness of the fp32 sums: a work unit sums at most 2^24 products per output; past
# that the inner range is split and the parts' int32 partial counts are added
# --------------------------------------------------------------------------
@pytest.mark.parametrize("polarity", [0, 1])
def test_exact_at_the_bound(dev, oracle_mod, polarity):
    rng = np.random.default_rng(171 + polarity)
    K, L = 65536, 256                          # K * L = 2^24 exactly: one unit may hold it all
    g = W.random_gemm(rng, 1, 3, 5, K, L, polarity, 171, L_lo=L)
    # saturated operands drive the counts to their extremes (|2X - K L| up to K L)
    g.A[0, 0] = 127
    g.B[0, 0] = 127 if polarity == 0 else -127
    g.A[0, 1] = -127
    _note("at K*L = 2^24, polarity %d" % polarity)
    out, cnt = _run(g, dev)
    _compare(g, 0, np.arange(g.M), np.arange(g.N), out, cnt, oracle_mod, "bound")


PAST_BOUND = [
    # M, N, K, L_max, rng: every GEMM variant past K * L_max = 2^24: fragments
    # from int8 rows (N <= 128), 128-row planes (M <= 128), int8 chunks in 256 x 256 and in
    # 256 x 64 blocks, and with C-BSG the 256-row and 128-row planes GEMMs
    # (the planes cases sit just past the bound: their planes take (M + N) K L / 2 bytes)
    (3, 5, 65536, 512, 0),
    (3, 129, 4128, 4096, 0),
    (300, 300, 16384, 2048, 0),
    (300, 17, 16384, 2048, 0),
    (200, 200, 65600, 256, 1),
    (3, 5, 65600, 256, 1),
]


@pytest.mark.parametrize("polarity", [0, 1])
@pytest.mark.parametrize("case", PAST_BOUND, ids=[str(c) for c in PAST_BOUND])
def test_exact_past_the_bound(dev, oracle_mod, case, polarity):
    """Saturated rows and columns: every product +1 (or -1), so an unsplit fp32 sum would
    pass 2^24 and round; the counts must still be exact.  Rows of full length and a few
    shorter ones; the oracle on sampled rows and columns (B's streams of every column would
    not fit in memory)."""
    M, N, K, L_max, rng_kind = case
    seed = 181 + polarity
    rng = np.random.default_rng(seed + M + N)
    g = W.random_gemm(rng, 1, M, N, K, L_max, polarity, seed, L_lo=L_max - 40)
    g.L[0, :2] = L_max
    g.A[0, 0] = 127
    g.A[0, 1] = -127
    g.B[0, 0] = 127
    g.B[0, N - 1] = -127
    _note("past the bound %s polarity %d" % (case, polarity))
    out, cnt = _run(g, dev, rng=rng_kind)
    rows = np.union1d([0, 1, M - 1], rng.choice(M, size=min(M, 3), replace=False))
    cols = np.union1d([0, N - 1], rng.choice(N, size=min(N, 4), replace=False))
    _compare(g, 0, rows, cols, out, cnt, oracle_mod, "past bound %s pol%d" % (case, polarity), rng=rng_kind)
    if polarity == 0:
        assert cnt[0, 0, 0] == K * L_max           # every XNOR is 1 (cycles and elements)
