"""The oracle's full-size digests (CPU): present for every workload, written by this oracle
for these inputs, covering every row, and reproduced by the oracle on a few blocks."""
import numpy as np
import pytest

import fullsize_digests as FD
import workloads as W

NAMES = ["vitb16_fc1_L128", "vitb16_fc1_mp64", "ditxl2_proj_mlp_group96", "vitl14_336_qk_mlp",
         "vitl14_compensator_L256", "vitl14_336_attn_av"]
CASES = [(n, False) for n in NAMES] + [("vitb16_fc1_L128", True)]


@pytest.mark.parametrize("name,cbsg", CASES, ids=[n + ("_cbsg" if c else "") for n, c in CASES])
def test_digests_cover_every_row_of_current_inputs(name, cbsg):
    dg = FD.load(name, cbsg)
    assert dg["oracle"] == FD.oracle_source_digest(), "stale digests: rerun make_fullsize_digests.py"
    w = W.WORKLOADS[name]()
    assert sorted(dg["inputs"]) == sorted(g.name for g in w.gemms)
    for g in w.gemms:
        assert FD.input_digests(g) == dg["inputs"][g.name]
        seen = {}
        for b, r0, r1, _ in dg["blocks"][g.name]:
            seen.setdefault(b, []).append((r0, r1))
        assert sorted(seen) == list(range(g.batch))
        for b, spans in seen.items():
            spans.sort()
            assert spans[0][0] == 0 and spans[-1][1] == g.M
            assert all(spans[k][1] == spans[k + 1][0] for k in range(len(spans) - 1))


@pytest.mark.parametrize("name,gname,b,r0", [
    ("vitl14_compensator_L256", "compensator", 0, 0),
    ("vitl14_compensator_L256", "compensator", 15, 8192),
    ("vitl14_336_attn_av", "attn_av", 0, 0),
    ("vitl14_336_qk_mlp", "attn_qk", 127, 512),
])
def test_oracle_reproduces_sampled_blocks(oracle_mod, name, gname, b, r0):
    if name == "vitl14_336_qk_mlp":
        w = W.vitl14_336_qk_mlp(mlp=False)
    else:
        w = W.WORKLOADS[name]()
    g = [x for x in w.gemms if x.name == gname][0]
    dg = FD.load(name)
    blk = [x for x in dg["blocks"][gname] if x[0] == b and x[1] == r0][0]
    r1 = blk[2]
    bB = 0 if g.B.shape[0] == 1 else b
    c, _ = oracle_mod.sc_gemm(g.A[b][r0:r1], g.B[bB], g.sA[b][r0:r1], g.sB[bB], g.L[b][r0:r1],
                              g.L_max, g.polarity, g.seed, want_out=False)
    assert FD.block_digest(c) == blk[3]
