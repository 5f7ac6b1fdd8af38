"""Reading the oracle's digests of the full-size count matrices (tests/golden/fullsize/).

The files are written by tests/golden/make_fullsize_digests.py, which calls only the CPU
oracle and the seeded workload generators.  Each block line holds the sha256 (first 32 hex
digits) of the int32 little-endian bytes of count rows [r0, r1) of one batch entry.
"""
import hashlib
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
DIR = os.path.join(HERE, "golden", "fullsize")


def path(name, cbsg=False):
    return os.path.join(DIR, "%s%s.txt" % (name, "_cbsg" if cbsg else ""))


def load(name, cbsg=False):
    """{"oracle": sha, "inputs": {gemm: {key: sha}}, "blocks": {gemm: [(b, r0, r1, sha)]}}"""
    d = {"oracle": None, "inputs": {}, "blocks": {}}
    with open(path(name, cbsg)) as f:
        for ln in f:
            t = ln.split()
            if not t or t[0].startswith("#"):
                continue
            if t[0] == "oracle_source_sha256":
                d["oracle"] = t[1]
            elif t[0] == "input":
                d["inputs"][t[1]] = dict(zip(t[2::2], t[3::2]))
            elif t[0] == "block":
                d["blocks"].setdefault(t[1], []).append((int(t[2]), int(t[3]), int(t[4]), t[5]))
    return d


def sha(a, n=64):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()[:n]


def oracle_source_digest():
    with open(os.path.join(ROOT, "oracle", "sc_oracle.c"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def input_digests(g):
    return {k: sha(v) for k, v in (("A", g.A), ("B", g.B), ("sA", g.sA), ("sB", g.sB), ("L", g.L))}


def block_digest(counts_rows):
    return sha(np.asarray(counts_rows, dtype="<i4"), 32)
