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


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sc_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert {"sc_gemm", "sc_gemm_workspace_size", "sc_gemm_status", "sc_strerror"} <= set(names)
    so = ctypes.CDLL(lib.LIB_PATH)
    for n in names:
        assert hasattr(so, n), n


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
  F(strideSA) F(strideSB) F(strideL) F(L_max) F(polarity) F(rng) F(L_hint) F(engine)
  F(reserved) F(seed)
  F(prof_event_begin) F(prof_event_end)
  printf("L_MAX %d K_LIMIT %d\\n", SC_L_MAX_LIMIT, SC_K_LIMIT);
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
    ("engine", 3, -10), ("engine", -1, -10), ("reserved", 1, -10),
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
    # on the VALU engine C-BSG keeps a count table but no marginals of B
    lfsr = lib.sc_gemm_workspace_size(_desc(lib, L_max=256, N=4096, ldo=4096, engine=1))
    cbsg = lib.sc_gemm_workspace_size(_desc(lib, rng=1, L_max=256, N=4096, ldo=4096, engine=1))
    assert cbsg < lfsr


def test_mfma_engine_exactness_bound(lib):
    # fp32 counts are exact only while K * L_max <= 2^24: an explicit MFMA request past
    # it is refused, AUTO takes the VALU engine there
    so = lib.load()
    n = ctypes.c_size_t(0)
    big = _desc(lib, K=65536, lda=65536, ldb=65536, L_max=512, engine=lib.SC_ENGINE_MFMA)
    assert so.sc_gemm_workspace_size(ctypes.byref(big), ctypes.byref(n)) == lib.SC_ERR_ENGINE
    for eng in (lib.SC_ENGINE_AUTO, lib.SC_ENGINE_VALU):
        ok = _desc(lib, K=65536, lda=65536, ldb=65536, L_max=512, engine=eng)
        assert lib.sc_gemm_workspace_size(ok) > 0
    at = _desc(lib, K=65536, lda=65536, ldb=65536, L_max=256, engine=lib.SC_ENGINE_MFMA)
    assert lib.sc_gemm_workspace_size(at) > 0


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
