"""The C-ABI library loads, exports every declared symbol and rejects bad arguments
before any HIP call (CPU only: nothing here launches a kernel)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scgemm.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2609_32922_amd._lib as L
    if not os.path.exists(L.LIB_PATH):
        from paper_2609_32922_amd import build
        build.build()
    return L


def _declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sc_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert {"sc_gemm", "sc_gemm_workspace_size", "sc_gemm_status", "sc_strerror"} <= set(names)
    so = ctypes.CDLL(lib.LIB_PATH)
    for n in names:
        assert hasattr(so, n), n


def test_every_header_is_served_by_a_library(lib):
    # include/scgemm.h by libscgemm, include/scpeak.h by libscpeak (the benchmark's VALU
    # peak measurement); no other header
    from paper_2609_32922_amd import peak
    served = {"scgemm.h": lib.LIB_PATH, "scpeak.h": peak.LIB_PATH}
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == sorted(served)
    for h, path in served.items():
        so = ctypes.CDLL(path)
        names = _declared_functions(os.path.join(ROOT, "include", h))
        assert names
        for n in names:
            assert hasattr(so, n), (h, n)


def test_peak_result_layout_matches_header(tmp_path):
    from paper_2609_32922_amd import peak
    src = tmp_path / "peak.c"
    src.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "scpeak.h"
#define F(f) printf("%s %zu\\n", #f, offsetof(sc_peak_result, f));
int main(void) {
  printf("size %zu\\n", sizeof(sc_peak_result));
  F(seconds) F(lane_ops_per_s) F(bitops_per_s) F(clock_hz) F(cus) F(waves_per_simd)
  return 0;
}
""")
    exe = tmp_path / "peak"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = dict(ln.split()[:2] for ln in subprocess.run([str(exe)], capture_output=True, text=True,
                                                         check=True).stdout.split("\n") if ln)
    R = peak.ScPeakResult
    assert int(got["size"]) == ctypes.sizeof(R)
    for name, _ in R._fields_:
        assert int(got[name]) == getattr(R, name).offset, name
    # argument errors return before any HIP call
    so = peak.load()
    r = peak.ScPeakResult()
    assert so.sc_peak_valu_bitop(0, 10, ctypes.byref(r)) == -1
    assert so.sc_peak_valu_bitop(9, 10, ctypes.byref(r)) == -1
    assert so.sc_peak_valu_bitop(1, 0, ctypes.byref(r)) == -1
    assert so.sc_peak_valu_bitop(1, 10, None) == -1


def test_desc_layout_matches_header(lib, tmp_path):
    src = tmp_path / "layout.c"
    src.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "scgemm.h"
#define F(f) printf("%s %zu\\n", #f, offsetof(sc_gemm_desc, f));
int main(void) {
  printf("size %zu\\n", sizeof(sc_gemm_desc));
  F(batch) F(M) F(N) F(K) F(lda) F(ldb) F(ldo) F(strideA) F(strideB) F(strideO)
  F(strideSA) F(strideSB) F(strideL) F(L_max) F(polarity) F(rng) F(L_hint)
  F(reserved) F(seed)
  F(prof_event_begin) F(prof_event_end)
  printf("L_MAX %d K_LIMIT %d KL_LIMIT %lld\\n", SC_L_MAX_LIMIT, SC_K_LIMIT, (long long)SC_KL_LIMIT);
  return 0;
}
""")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    lines = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = dict(ln.split()[:2] for ln in lines if ln and not ln.startswith("L_MAX"))
    D = lib.ScGemmDesc
    assert int(got["size"]) == ctypes.sizeof(D)
    for name, _ in D._fields_:
        assert int(got[name]) == getattr(D, name).offset, name
    last = [ln for ln in lines if ln.startswith("L_MAX")][0].split()
    assert int(last[1]) == lib.SC_L_MAX_LIMIT and int(last[3]) == lib.SC_K_LIMIT
    assert int(last[5]) == lib.SC_KL_LIMIT


def _desc(lib, **kw):
    d = lib.ScGemmDesc()
    d.batch, d.M, d.N, d.K = 1, 64, 64, 256
    d.lda, d.ldb, d.ldo = 256, 256, 64
    d.L_max, d.polarity, d.rng, d.L_hint, d.seed = 64, 0, 0, 0, 0
    for k, v in kw.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("field,value,code", [
    ("M", -1, -2), ("K", -5, -2), ("batch", -1, -2), ("K", (1 << 20) + 1, -2),
    ("L_max", 0, -3), ("L_max", 4097, -3), ("polarity", 2, -4), ("rng", 2, -5), ("rng", -1, -5),
    ("L_hint", 65, -3), ("L_hint", -1, -3), ("lda", 255, -9), ("ldo", 63, -9), ("strideA", -1, -9),
    ("reserved", 1, -10), ("reserved", -1, -10),
])
def test_workspace_size_rejects_bad_desc(lib, field, value, code):
    n = ctypes.c_size_t(0)
    so = lib.load()
    d = _desc(lib, **{field: value})
    assert so.sc_gemm_workspace_size(ctypes.byref(d), ctypes.byref(n)) == code


def test_cbsg_length_limit(lib):
    # the Sobol-8 sequences have period 256: longer C-BSG streams are rejected
    assert lib.sc_gemm_workspace_size(_desc(lib, rng=1, L_max=256)) > 0
    so = lib.load()
    n = ctypes.c_size_t(0)
    d = _desc(lib, rng=1, L_max=257, L_hint=0)
    assert so.sc_gemm_workspace_size(ctypes.byref(d), ctypes.byref(n)) == lib.SC_ERR_LEN


def test_exactness_bound_splits(lib):
    # fp32 sums stay exact for 2^24 products per part: past that the inner range is split
    # (int32 partial sums, more workspace), and past 8 parts (K * L_max > 2^27) refused
    so = lib.load()
    n = ctypes.c_size_t(0)
    # 4096 x 4096: 256 tiles of 256 x 256, one round on 256 CUs, so nothing is split at
    # K * L_max = 2^24; one chunk more and every tile is split in two
    at = lib.sc_gemm_workspace_size(_desc(lib, M=4096, N=4096, ldo=4096, K=4096, lda=4096, ldb=4096,
                                          L_max=4096))
    past = lib.sc_gemm_workspace_size(_desc(lib, M=4096, N=4096, ldo=4096, K=4128, lda=4128, ldb=4128,
                                            L_max=4096))
    assert past >= at + 2 * 4096 * 4096 * 4
    for M, N in ((64, 64), (64, 300), (300, 300), (300, 64)):
        top = _desc(lib, M=M, N=N, ldo=N, K=32768, lda=32768, ldb=32768, L_max=4096)
        assert lib.sc_gemm_workspace_size(top) > 0
        over = _desc(lib, M=M, N=N, ldo=N, K=32769, lda=32769, ldb=32769, L_max=4096)
        assert so.sc_gemm_workspace_size(ctypes.byref(over), ctypes.byref(n)) == lib.SC_ERR_SHAPE
        cb = _desc(lib, M=M, N=N, ldo=N, K=524288, lda=524288, ldb=524288, L_max=256, rng=1)
        assert lib.sc_gemm_workspace_size(cb) > 0


def test_workspace_size_values(lib):
    d = _desc(lib)
    n1 = lib.sc_gemm_workspace_size(d)
    d2 = _desc(lib, L_max=128)
    n2 = lib.sc_gemm_workspace_size(d2)
    assert 0 < n1 < n2 and n1 % 256 == 0
    d3 = _desc(lib, polarity=1)
    assert lib.sc_gemm_workspace_size(d3) > 0
    so = lib.load()
    assert so.sc_gemm_workspace_size(ctypes.byref(d), None) == lib.SC_ERR_NULL
    assert so.sc_gemm_workspace_size(None, ctypes.byref(ctypes.c_size_t())) == lib.SC_ERR_NULL


def test_sc_gemm_argument_errors_before_any_hip_call(lib):
    d = _desc(lib)
    fake = 1 << 40                      # never dereferenced: every call below returns early
    args = [fake] * 7
    assert lib.sc_gemm(d, 0, *args[1:6], 0, fake, 1 << 30, 0) == lib.SC_ERR_NULL
    assert lib.sc_gemm(d, fake, fake, fake, fake, fake, 0, 0, fake, 1 << 30, 0) == lib.SC_ERR_NULL
    need = lib.sc_gemm_workspace_size(d)
    assert lib.sc_gemm(d, *args[:6], 0, fake, need - 1, 0) == lib.SC_ERR_WORKSPACE
    assert lib.sc_gemm(d, *args[:6], 0, 0, need, 0) == lib.SC_ERR_WORKSPACE
    assert lib.sc_gemm(d, *args[:6], 0, fake + 16, need, 0) == lib.SC_ERR_WORKSPACE  # misaligned
    bad = _desc(lib, polarity=5)
    assert lib.sc_gemm(bad, *args[:6], 0, fake, need, 0) == lib.SC_ERR_POLARITY
    so = lib.load()
    assert so.sc_gemm(None, *([None] * 8), 0, None) == lib.SC_ERR_NULL


def test_comparator_sequence_argument_errors(lib):
    fake = 1 << 40
    assert lib.sc_comparator_sequence(0, 0, 0, 16, 0, 0) == lib.SC_ERR_NULL
    assert lib.sc_comparator_sequence(0, 2, 0, 16, fake, 0) == lib.SC_ERR_RNG
    assert lib.sc_comparator_sequence(0, 0, 2, 16, fake, 0) == lib.SC_ERR_RNG
    assert lib.sc_comparator_sequence(0, 0, 0, 0, fake, 0) == lib.SC_ERR_LEN
    assert lib.sc_comparator_sequence(0, 0, 0, 4097, fake, 0) == lib.SC_ERR_LEN
    assert lib.sc_comparator_sequence(0, 1, 1, 257, fake, 0) == lib.SC_ERR_LEN
    assert lib.sc_gemm_status(0, 0) == lib.SC_ERR_NULL


def test_strerror_and_version(lib):
    for code in range(-10, 1):
        assert lib.strerror(code).startswith("SC_")
    assert "unknown" in lib.strerror(-100)
    assert lib.sc_version() >= 10000


def test_product_package_does_not_import_oracle():
    # the binding and the library never reach the CPU oracle
    pkg = os.path.join(ROOT, "paper_2609_32922_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "sc_oracle" not in text, f
