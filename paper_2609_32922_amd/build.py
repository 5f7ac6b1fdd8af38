"""Build libscgemm.so (the SC GEMM library) and libscpeak.so (its VALU peak
microbenchmark, used by the benchmark only) for gfx950 with hipcc, in-tree next to this
file.

    python -m paper_2609_32922_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["sc_kernels.hip", "sc_mfma.hip", "sc_frontend.hip", "sc_api.hip"]
OUT = os.path.join(HERE, "libscgemm.so")
PEAK_SOURCES = ["sc_peak.hip"]
PEAK_OUT = os.path.join(HERE, "libscpeak.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed-FP32 instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _compile(sources, out, verbose):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + HIPCC_FLAGS + [os.path.join(CSRC, s) for s in sources] + ["-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(ln for ln in (res.stdout + res.stderr).splitlines()
                    if "packed-fp32-ops" not in ln)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n%s\n%s" % (" ".join(cmd), msg))
    if verbose and msg.strip():
        print(msg)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """Compile libscgemm.so and libscpeak.so; always recompiles.  Returns libscgemm's path."""
    _compile(PEAK_SOURCES, PEAK_OUT, verbose)
    return _compile(SOURCES, OUT, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
