"""Write the golden fixtures of this folder from the CPU oracle only.

Run from the repository root:  python tests/golden/make_golden.py
The fixtures freeze the oracle's comparator sequences (LFSR reading of Sec. A.1),
its boundary tables (V = 257 boundaries, Sec. 4.2) and the count matrix of the
64x256x64 bipolar workload, so that any later change to the oracle's arithmetic
shows up as a diff that has to be justified by the paper.
"""
import hashlib
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads  # noqa: E402


def main():
    with open(os.path.join(HERE, "lfsr_draws.txt"), "w") as f:
        f.write("# seed op state  first 32 comparator draws r_0..r_31 (uint8)\n")
        for seed in range(5):
            for op in (0, 1):
                st = oracle.seed_state(seed, op)
                r = oracle.comparator_sequence(seed, op, 32)
                f.write("%d %d %08x %s\n" % (seed, op, st, " ".join(str(int(x)) for x in r)))
    with open(os.path.join(HERE, "beta_tables.txt"), "w") as f:
        f.write("# q beta_bipolar(q) beta_unipolar(q)\n")
        for q in range(-127, 128):
            f.write("%d %d %d\n" % (q, oracle.beta_bipolar(q), oracle.beta_unipolar(q)))
    w = workloads.bipolar_64x256x64()
    g = w.gemms[0]
    c, o = oracle.sc_gemm(g.A[0], g.B[0], g.sA[0], g.sB[0], g.L[0], g.L_max, g.polarity, g.seed)
    with open(os.path.join(HERE, "bipolar_64x256x64_counts.txt"), "w") as f:
        f.write("# workload bipolar_64x256x64_L64 (seed 0): XNOR count matrix X[64][64]\n")
        f.write("# sha256(int32 little-endian row-major) %s\n"
                % hashlib.sha256(c.astype("<i4").tobytes()).hexdigest())
        for row in c:
            f.write(" ".join(str(int(x)) for x in row) + "\n")


if __name__ == "__main__":
    main()
