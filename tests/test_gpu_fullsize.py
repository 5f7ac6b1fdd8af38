"""Every output of the full-size workloads against the oracle (GPU, through the C ABI).

The oracle's count matrices of these workloads are too large to recompute at test time
(up to 1e13 materialised stream bits per workload), so tests/golden/make_fullsize_digests.py
computed them once, from the oracle alone, and stored a sha256 per block of 256 rows.
Here the library runs each GEMM in the launch configuration the benchmark times (the same
L_hint), and:
  * the inputs are checked to be the ones the oracle saw (sha256 of A, B, scales, lengths);
  * every block of the count matrix must hash to the oracle's digest: counts bit-exact
    for every output (Eq. (1) counts: bipolar XNOR counts, unipolar signed AND counts);
  * every decoded float is compared with the oracle's Eq. (1) decode of those counts
    (float64): within 1e-6 relative, exact zeros where the oracle has them.
"""
import sys

import numpy as np
import pytest

import fullsize_digests as FD
import workloads as W

pytestmark = pytest.mark.gpu

REL_TOL = 1e-6

CASES = [("vitb16_fc1_L128", False), ("vitb16_fc1_mp64", False), ("ditxl2_proj_mlp_group96", False),
         ("vitl14_336_qk_mlp", False), ("vitl14_compensator_L256", False), ("vitl14_336_attn_av", False),
         ("vitb16_fc1_L128", True)]


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


def _run(g, dev, rng):
    import torch
    import paper_2609_32922_amd as scg
    A, sA, B, sB, L = (torch.from_numpy(np.ascontiguousarray(x)).to(dev)
                       for x in (g.A, g.sA, g.B, g.sB, g.L))
    out, cnt = scg.gemm(A, sA, B, sB, L, L_max=g.L_max, polarity=g.polarity, seed=g.seed,
                        want_counts=True, check_status=True, rng=rng,
                        L_hint=int(round(float(g.L.mean()))))
    torch.cuda.synchronize()
    o, c = out.cpu().numpy(), cnt.cpu().numpy()
    del A, sA, B, sB, L, out, cnt
    torch.cuda.empty_cache()
    return o, c


@pytest.mark.parametrize("name,cbsg", CASES, ids=[n + ("_cbsg" if c else "") for n, c in CASES])
def test_every_output_matches_oracle(dev, oracle_mod, name, cbsg):
    dg = FD.load(name, cbsg)
    assert dg["oracle"] == FD.oracle_source_digest(), \
        "the digests were written by another version of the oracle: rerun make_fullsize_digests.py"
    w = W.WORKLOADS[name]()
    for g in w.gemms:
        assert FD.input_digests(g) == dg["inputs"][g.name], g.name + ": inputs differ from the oracle's"
        _note("%s/%s every output, %s" % (name, g.name, "C-BSG" if cbsg else "LFSR"))
        out, cnt = _run(g, dev, 1 if cbsg else 0)
        blocks = dg["blocks"][g.name]
        assert sum(r1 - r0 for _, r0, r1, _ in blocks) == g.batch * g.M
        bad = [(b, r0, r1) for b, r0, r1, h in blocks if FD.block_digest(cnt[b, r0:r1]) != h]
        assert not bad, "%s/%s: %d of %d row blocks differ from the oracle, first %s" % (
            name, g.name, len(bad), len(blocks), bad[0])
        worst = 0.0
        for b in range(g.batch):
            bB = 0 if g.B.shape[0] == 1 else b
            ref = oracle_mod.decode(cnt[b], g.sA[b], g.sB[bB], g.L[b], g.K, g.polarity)
            o = out[b].astype(np.float64)
            zero = ref == 0.0
            assert np.all(o[zero] == 0.0), "%s/%s b%d: expected exact zeros" % (name, g.name, b)
            if (~zero).any():
                rel = np.abs(o[~zero] - ref[~zero]) / np.abs(ref[~zero])
                worst = max(worst, float(rel.max()))
        assert worst <= REL_TOL, "%s/%s: max relative error %.3g" % (name, g.name, worst)
        _note("%s/%s: %d outputs exact, max rel err %.2g" % (name, g.name, cnt.size, worst))
