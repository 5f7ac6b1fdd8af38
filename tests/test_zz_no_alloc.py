"""The allocation-free entry point sc_gemm_noalloc against sc_gemm, through the C ABI.

Both run the same kernels, so counts and decoded floats must agree bit for bit (stricter
than the 1e-6 relative bar of the oracle comparisons); two calls in a row, the second on a
smaller problem, so that it runs on the contents the first call left in the library's
array.  The argument checks run on the CPU."""
import ctypes
import sys

import numpy as np
import pytest

import workloads as W


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


def _both(g, dev):
    import torch
    import paper_2609_32922_amd as scg
    A, sA, B, sB, L = (torch.from_numpy(np.ascontiguousarray(x)).to(dev)
                       for x in (g.A, g.sA, g.B, g.sB, g.L))
    o1, c1 = scg.gemm(A, sA, B, sB, L, L_max=g.L_max, polarity=g.polarity, seed=g.seed,
                      want_counts=True, check_status=True)
    d = scg.make_desc(A, B, g.L_max, g.polarity, g.seed)
    o2 = torch.full_like(o1, float("nan"))
    c2 = torch.full_like(c1, -7)
    st = torch.full((1,), -1, dtype=torch.int32, device=dev)
    sh = int(torch.cuda.current_stream().cuda_stream)
    rc = scg.sc_gemm_noalloc(d, A.data_ptr(), sA.data_ptr(), B.data_ptr(), sB.data_ptr(), L.data_ptr(),
                             o2.data_ptr(), c2.data_ptr(), st.data_ptr(), sh)
    assert rc == 0, scg.strerror(rc)
    torch.cuda.synchronize()
    return (o1.cpu().numpy(), c1.cpu().numpy(), o2.cpu().numpy(), c2.cpu().numpy(), int(st.item()))


@pytest.mark.gpu
def test_noalloc_matches_sc_gemm_twice(dev):
    import paper_2609_32922_amd as scg
    w = W.vitb16_fc1_L128()                                   # 35 MiB of workspace
    cases = [("vitb16_fc1_L128", w.gemms[0]),
             ("300x260x100 per-row L", W.random_gemm(np.random.default_rng(3), 1, 300, 260, 100, 96, 1, 33))]
    for name, g in cases:
        d = scg.make_desc(*(__import__("torch").from_numpy(x) for x in (g.A, g.B)), g.L_max, g.polarity, g.seed)
        assert scg.sc_gemm_workspace_size(d) <= scg.SC_NOALLOC_WORKSPACE_BYTES
        _note("no-alloc entry point: " + name)
        o1, c1, o2, c2, st = _both(g, dev)
        assert st == 0
        assert np.array_equal(c1, c2), name + ": counts differ"
        assert np.array_equal(o1.view(np.uint32), o2.view(np.uint32)), name + ": decoded floats differ"


@pytest.mark.gpu
def test_noalloc_reports_bad_lengths(dev):
    import paper_2609_32922_amd as scg
    import torch
    g = W.random_gemm(np.random.default_rng(5), 1, 50, 20, 16, 32, 0, 41)
    g.L[0, 3] = 33
    A, sA, B, sB, L = (torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in (g.A, g.sA, g.B, g.sB, g.L))
    d = scg.make_desc(A, B, g.L_max, g.polarity, g.seed)
    out = torch.empty((1, 50, 20), dtype=torch.float32, device=dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    _note("no-alloc entry point: bad length")
    rc = scg.sc_gemm_noalloc(d, A.data_ptr(), sA.data_ptr(), B.data_ptr(), sB.data_ptr(), L.data_ptr(),
                             out.data_ptr(), 0, st.data_ptr(), int(torch.cuda.current_stream().cuda_stream))
    assert rc == 0
    torch.cuda.synchronize()
    assert int(st.item()) & 1


def test_noalloc_argument_errors_before_any_hip_call():
    import paper_2609_32922_amd._lib as L
    d = L.ScGemmDesc()
    d.batch, d.M, d.N, d.K = 1, 6400, 6400, 4096
    d.lda, d.ldb, d.ldo = 4096, 4096, 6400
    d.L_max = 512
    fake = 1 << 40                          # never dereferenced: every call returns early
    assert L.sc_gemm_workspace_size(d) > L.SC_NOALLOC_WORKSPACE_BYTES
    assert L.sc_gemm_noalloc(d, *([fake] * 6), 0, 0, 0) == L.SC_ERR_WORKSPACE
    assert L.sc_gemm_noalloc(d, 0, *([fake] * 5), 0, 0, 0) == L.SC_ERR_NULL
    d.reserved = 1
    assert L.sc_gemm_noalloc(d, *([fake] * 6), 0, 0, 0) == L.SC_ERR_RESERVED
    so = L.load()
    assert so.sc_gemm_noalloc(None, *([None] * 8), None) == L.SC_ERR_NULL
