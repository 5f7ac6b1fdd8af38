"""Write digests of the oracle's full count matrices of the full-size workloads.

Run from the repository root (long: every stream of every workload is materialised):

    python tests/golden/make_fullsize_digests.py [--threads N] [--cbsg] [workload ...]

For every GEMM and batch entry of a workload the CPU oracle computes the whole count
matrix (Eq. (1): XNOR counts for bipolar, signed AND counts for unipolar
sign-magnitude), block by block of ROWS rows, and this script stores the sha256 of each
block's int32 little-endian row-major bytes, together with the sha256 of the workload's
inputs and of the oracle's C source.  The GPU test hashes the library's counts the same
way, so every output of every workload is compared bit for bit without running the
oracle at test time.  Nothing here reads anything the HIP library wrote: the only
inputs are the seeded generators in ``workloads`` and the oracle.
"""
import argparse
import hashlib
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads  # noqa: E402

ROWS = 256
OUT_DIR = os.path.join(HERE, "fullsize")
DEFAULT = ["vitb16_fc1_L128", "vitb16_fc1_mp64", "ditxl2_proj_mlp_group96", "vitl14_336_qk_mlp",
           "vitl14_compensator_L256", "vitl14_336_attn_av"]


def sha(a: np.ndarray, n: int = 64) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()[:n]


def oracle_source_digest() -> str:
    with open(os.path.join(ROOT, "oracle", "sc_oracle.c"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def digest_path(name: str, cbsg: bool) -> str:
    return os.path.join(OUT_DIR, "%s%s.txt" % (name, "_cbsg" if cbsg else ""))


def input_digests(g) -> str:
    return " ".join("%s %s" % (k, sha(v.astype(v.dtype.newbyteorder("<"))))
                    for k, v in (("A", g.A), ("B", g.B), ("sA", g.sA), ("sB", g.sB), ("L", g.L)))


def run(name: str, cbsg: bool, threads: int):
    w = workloads.WORKLOADS[name]()
    ref = oracle.sc_gemm_cbsg if cbsg else oracle.sc_gemm
    lines = ["# written by tests/golden/make_fullsize_digests.py from the CPU oracle only",
             "# workload %s rng %s rows_per_block %d" % (w.name, "sobol8_cbsg" if cbsg else "lfsr32", ROWS),
             "oracle_source_sha256 %s" % oracle_source_digest()]
    t0 = time.time()
    for g in w.gemms:
        lines.append("input %s %s" % (g.name, input_digests(g)))
        for b in range(g.batch):
            bB = 0 if g.B.shape[0] == 1 else b
            for r0 in range(0, g.M, ROWS):
                r1 = min(g.M, r0 + ROWS)
                c, _ = ref(g.A[b][r0:r1], g.B[bB], g.sA[b][r0:r1], g.sB[bB], g.L[b][r0:r1],
                           g.L_max, g.polarity, g.seed, nthreads=threads, want_out=False)
                lines.append("block %s %d %d %d %s" % (g.name, b, r0, r1, sha(c.astype("<i4"), 32)))
            print("%s %s batch %d/%d done, %.0f s" % (name, g.name, b + 1, g.batch, time.time() - t0),
                  flush=True)
    os.makedirs(OUT_DIR, exist_ok=True)
    with open(digest_path(name, cbsg), "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    p = argparse.ArgumentParser()
    p.add_argument("workloads", nargs="*", default=DEFAULT)
    p.add_argument("--threads", type=int, default=0)
    p.add_argument("--cbsg", action="store_true", help="Sobol-8 C-BSG streams instead of the LFSR")
    a = p.parse_args()
    for name in a.workloads:
        run(name, a.cbsg, a.threads)


if __name__ == "__main__":
    main()
