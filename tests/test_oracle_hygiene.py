"""CPU hygiene of the oracle and of the library's host code: the oracle gives identical
results on 1 and on N threads, and both run clean under AddressSanitizer and
UndefinedBehaviorSanitizer (host code only; nothing here runs on a GPU)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.parametrize("cbsg", [False, True])
@pytest.mark.parametrize("polarity", [0, 1])
def test_oracle_one_thread_equals_many(oracle_mod, polarity, cbsg):
    rng = np.random.default_rng(7 + polarity + 2 * cbsg)
    g = W.random_gemm(rng, 1, 37, 29, 45, 96, polarity, 5)
    g.L[0, :3] = 0
    ref = oracle_mod.sc_gemm_cbsg if cbsg else oracle_mod.sc_gemm
    args = (g.A[0], g.B[0], g.sA[0], g.sB[0], g.L[0], g.L_max, polarity, g.seed)
    c1, o1 = ref(*args, nthreads=1)
    for n in (2, 5, 8):
        cn, on = ref(*args, nthreads=n)
        assert np.array_equal(c1, cn) and np.array_equal(o1.view(np.uint64), on.view(np.uint64))


def _run(cmd, **kw):
    return subprocess.run(cmd, capture_output=True, text=True, **kw)


@pytest.mark.slow
def test_oracle_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_asan"
    src = os.path.join(HERE, "sanitize", "oracle_driver.c")
    r = _run(["gcc", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
              "-fno-sanitize-recover=all", "-std=c11", src, os.path.join(ROOT, "oracle", "sc_oracle.c"),
              "-o", str(exe)])
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", OMP_NUM_THREADS="4")
    r = _run([str(exe)], env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    assert "oracle driver ok" in r.stdout


HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


@pytest.mark.slow
@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_code_under_sanitizers(tmp_path):
    """The library's argument checks and workspace layout (check_desc, make_layout, the
    split choice) over many descriptors, host code instrumented, device code as usual; every
    call returns before anything would be enqueued, so no GPU is needed."""
    exe = tmp_path / "host_asan"
    csrc = os.path.join(ROOT, "paper_2609_32922_amd", "csrc")
    srcs = [os.path.join(csrc, s) for s in ("sc_kernels.hip", "sc_mfma.hip", "sc_frontend.hip", "sc_api.hip")]
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "sanitize", "host_driver.cpp")] + srcs + ["-o", str(exe)]
    r = _run(cmd)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:protect_shadow_gap=0", HIP_VISIBLE_DEVICES="")
    r = _run([str(exe)], env=env, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr
    assert "host driver ok" in r.stdout
