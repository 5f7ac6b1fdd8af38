"""GPU parity of the front end: int8 quantisation, per-row length policy, and the
whole device pipeline fp32 -> int8 -> lengths -> SC GEMM against the oracle's.

Quantised integers, scales and lengths are integer (or exactly reproduced fp32)
decisions taken in fp32 on both sides: compared bit for bit."""
import sys

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


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


def _t(x, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def test_quantize_rows_and_tensor(dev, oracle_mod):
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(3)
    X = rng.standard_normal((2, 150, 777)).astype(np.float32)
    X[:, :, 5] *= 30
    X[0, 7] = 0.0
    X[1, :, 100] = np.float32(1.5)        # ties after scaling are possible
    _note("quantize rows")
    Q, s, m = scg.quantize(_t(X, dev), per_tensor=False, want_rowmax=True)
    Q, s, m = Q.cpu().numpy(), s.cpu().numpy(), m.cpu().numpy()
    for b in range(2):
        Qr, sr, mr = oracle_mod.quantize_rows_fp32(X[b])
        assert np.array_equal(Q[b], Qr) and np.array_equal(s[b], sr) and np.array_equal(m[b], mr)
    _note("quantize tensor")
    Q, s, m = scg.quantize(_t(X, dev), per_tensor=True, want_rowmax=True)
    Q, s = Q.cpu().numpy(), s.cpu().numpy()
    for b in range(2):
        Qr, sr = oracle_mod.quantize_tensor_fp32(X[b])
        assert np.array_equal(Q[b], Qr) and np.array_equal(s[b], sr)


def test_quantize_full_size_against_host_quantiser(dev, oracle_mod):
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(1)
    X = rng.standard_normal((6304, 768)).astype(np.float32)
    X[:, rng.choice(768, 6, replace=False)] *= np.float32(20.0)
    _note("quantize 6304x768")
    Q, s, _ = scg.quantize(_t(X, dev))
    Q, s = Q.cpu().numpy(), s.cpu().numpy()
    Qh, sh = W.quantize_rows(X)
    assert np.array_equal(Q, Qh) and np.array_equal(s, sh)
    rows = [0, 1, 2, 4000, 6303]
    Qr, sr, _ = oracle_mod.quantize_rows_fp32(X[rows])
    assert np.array_equal(Q[rows], Qr) and np.array_equal(s[rows], sr)


def test_mp_lengths(dev, oracle_mod):
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(4)
    g = rng.gamma(2.0, 1.0, (3, 1001)).astype(np.float32)
    g[2] = np.float32(0.5)                # constant metric: shortest everywhere
    for tau, ladder in [([0.6, 0.3, 0.1], [192, 96, 48, 24]), ([], [77]),
                        ([0.5], [512, 8]), ([1.0, 0.0], [300, 200, 100])]:
        _note("mp_lengths %s %s" % (tau, ladder))
        L = scg.mp_lengths(_t(g, dev), tau, ladder).cpu().numpy()
        for b in range(3):
            assert np.array_equal(L[b], oracle_mod.mp_lengths_fp32(g[b], tau, ladder))


def test_mp_lengths_rejects_bad_ladders(dev):
    import torch
    import paper_2609_32922_amd as scg
    g = torch.ones(10, device=dev)
    for tau, ladder in [([0.5], [64, 64]), ([0.2, 0.5], [3, 2, 1]), ([1.5], [9, 3]), ([0.5], [9, -1])]:
        with pytest.raises(scg.ScError):
            scg.mp_lengths(g, tau, ladder)


def test_device_pipeline_end_to_end(dev, oracle_mod):
    """fp32 activations and weights -> device int8 + scales + row metric -> device
    lengths -> SC GEMM with the device length vector, against the oracle pipeline."""
    import torch
    import paper_2609_32922_amd as scg
    rng = np.random.default_rng(5)
    X = rng.standard_normal((300, 200)).astype(np.float32)
    X[:, 3] *= 12
    Wt = (rng.standard_normal((260, 200)) * 0.02).astype(np.float32)
    tau, ladder = [0.5, 0.25, 0.1], [160, 96, 48, 24]
    for pol in (0, 1):
        _note("pipeline polarity %d" % pol)
        qX, sX, mX = scg.quantize(_t(X, dev), want_rowmax=True)
        qW, sW, _ = scg.quantize(_t(Wt, dev), per_tensor=True)
        L = scg.mp_lengths(mX, tau, ladder)
        out, cnt = scg.gemm(qX, sX, qW, sW, L, L_max=160, polarity=pol, seed=11, want_counts=True,
                            check_status=True)
        torch.cuda.synchronize()
        oq, osx, om = oracle_mod.quantize_rows_fp32(X)
        ow, osw = oracle_mod.quantize_tensor_fp32(Wt)
        oL = oracle_mod.mp_lengths_fp32(om, tau, ladder)
        assert np.array_equal(L.cpu().numpy(), oL)
        c_ref, o_ref = oracle_mod.sc_gemm(oq, ow, osx, osw, oL, 160, pol, 11)
        assert np.array_equal(cnt.cpu().numpy(), c_ref)
        o = out.cpu().numpy().astype(np.float64)
        nz = o_ref != 0
        assert np.all(o[~nz] == 0)
        assert np.max(np.abs(o[nz] - o_ref[nz]) / np.abs(o_ref[nz])) <= 1e-6


def test_device_pipeline_with_threshold_table(dev, oracle_mod):
    """The policy of Sec. 4.4 with its calibrated-threshold table: per layer the table gives
    (thresholds, ladder) for the operator's timestep and layer bucket (or the operator-level
    fallback); the device turns the row metric into lengths, which drive the SC GEMM."""
    import os

    import torch
    import paper_2609_32922_amd as scg
    from paper_2609_32922_amd.thresholds import ThresholdTable, mp_lengths_from_table
    table = ThresholdTable.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                             "thresholds_synthetic.json"))
    rng = np.random.default_rng(6)
    X = rng.laplace(0.0, 1.0, (260, 120)).astype(np.float32)
    Wt = (rng.standard_normal((300, 120)) * 0.02).astype(np.float32)
    for op, t, layer, want in [("mlp_fc1", 3, 27, "bucket"), ("mlp_fc1", 40, 0, "operator"),
                               ("mlp_fc2", 12, 22, "bucket")]:
        _note("table pipeline %s t=%d layer=%d" % (op, t, layer))
        qX, sX, mX = scg.quantize(_t(X, dev), want_rowmax=True)
        qW, sW, _ = scg.quantize(_t(Wt, dev), per_tensor=True)
        L, thr = mp_lengths_from_table(mX, table, op, t, layer)
        assert thr.source == want
        L_max = thr.ladder[0]
        out, cnt = scg.gemm(qX, sX, qW, sW, L, L_max=L_max, polarity=1, seed=13, want_counts=True,
                            check_status=True)
        torch.cuda.synchronize()
        oq, osx, om = oracle_mod.quantize_rows_fp32(X)
        ow, osw = oracle_mod.quantize_tensor_fp32(Wt)
        oL = oracle_mod.mp_lengths_fp32(om, thr.tau, thr.ladder)
        assert np.array_equal(L.cpu().numpy(), oL)
        assert len(set(oL.tolist())) > 1
        c_ref, o_ref = oracle_mod.sc_gemm(oq, ow, osx, osw, oL, L_max, 1, 13)
        assert np.array_equal(cnt.cpu().numpy(), c_ref)
        o = out.cpu().numpy().astype(np.float64)
        nz = o_ref != 0
        assert np.all(o[~nz] == 0)
        assert np.max(np.abs(o[nz] - o_ref[nz]) / np.abs(o_ref[nz])) <= 1e-6
