"""The calibrated threshold table of the per-row mixed-precision policy (Sec. 4.4, "Threshold
fitting"): host-side loading and lookup, feeding ``sc_mp_lengths``.

The paper's calibration mode (out of scope here) writes a JSON table of metric thresholds,
keyed by operator, timestep bucket and layer-depth bucket, with an operator-level fallback
for buckets that are sparse.  At inference a layer looks up its thresholds
1 >= tau_1 >= ... >= tau_{K-1} >= 0 for its ladder L_1 > ... > L_K, and row i gets the first
level whose threshold its min-max normalised metric reaches, else the shortest.

Table format (the paper fixes only the keys; this layout is this library's):

    {
      "ladder": [256, 128, 64, 32],             default ladder, strictly decreasing
      "timestep_edges": [0, 10, 20, 50],        bucket b holds timesteps in [e_b, e_b+1)
      "layer_edges": [0, 8, 16, 28],            bucket b holds layer indices in [e_b, e_b+1)
      "min_rows": 64,                           optional: a bucket calibrated on fewer rows
                                                is sparse and falls back
      "entries": [
        {"operator": "mlp_fc1", "tau": [0.8, 0.5, 0.2]},                  operator level
        {"operator": "mlp_fc1", "timestep_bucket": 0, "layer_bucket": 2,
         "tau": [0.9, 0.6, 0.3], "rows": 512, "ladder": [...]},           one bucket
        ...
      ]
    }

An entry without bucket keys is the operator-level entry.  ``ladder`` in an entry overrides
the default.  Models without timesteps use one timestep bucket (``timestep_edges`` absent:
every timestep, including None, is bucket 0); likewise for layers.
"""
from __future__ import annotations

import bisect
import json
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

from ._lib import SC_L_MAX_LIMIT

MAX_LEVELS = 32          # SC_MP_MAX_LEVELS of the C ABI


@dataclass(frozen=True)
class Thresholds:
    tau: Tuple[float, ...]       # K-1 thresholds in [0, 1], non-increasing
    ladder: Tuple[int, ...]      # K lengths, strictly decreasing
    source: str                  # "bucket" or "operator" (where the lookup found them)


def _check(tau: Sequence[float], ladder: Sequence[int], where: str):
    if not 1 <= len(ladder) <= MAX_LEVELS:
        raise ValueError("%s: ladder needs 1..%d levels" % (where, MAX_LEVELS))
    if any(not isinstance(x, int) or x < 0 or x > SC_L_MAX_LIMIT for x in ladder):
        raise ValueError("%s: ladder lengths must be integers in [0, %d]" % (where, SC_L_MAX_LIMIT))
    if any(ladder[k] <= ladder[k + 1] for k in range(len(ladder) - 1)):
        raise ValueError("%s: ladder must be strictly decreasing" % where)
    if len(tau) != len(ladder) - 1:
        raise ValueError("%s: %d thresholds for %d levels" % (where, len(tau), len(ladder)))
    if any(not (0.0 <= t <= 1.0) for t in tau) or any(tau[k] < tau[k + 1] for k in range(len(tau) - 1)):
        raise ValueError("%s: thresholds must lie in [0, 1] and not increase" % where)


def _edges(x, name):
    if x is None:
        return None
    e = [int(v) for v in x]
    if len(e) < 2 or any(e[k] >= e[k + 1] for k in range(len(e) - 1)):
        raise ValueError("%s must hold at least two strictly increasing values" % name)
    return e


class ThresholdTable:
    """A loaded threshold table: ``lookup(operator, timestep, layer)``."""

    def __init__(self, doc: dict):
        self.ladder = tuple(int(x) for x in doc.get("ladder", ()))
        self.t_edges = _edges(doc.get("timestep_edges"), "timestep_edges")
        self.l_edges = _edges(doc.get("layer_edges"), "layer_edges")
        self.min_rows = int(doc.get("min_rows", 0))
        self._op: Dict[str, Thresholds] = {}
        self._bucket: Dict[Tuple[str, int, int], Tuple[Thresholds, Optional[int]]] = {}
        for n, e in enumerate(doc.get("entries", [])):
            op = e["operator"]
            ladder = tuple(int(x) for x in e.get("ladder", self.ladder))
            tau = tuple(float(x) for x in e["tau"])
            where = "entry %d (%s)" % (n, op)
            _check(tau, ladder, where)
            has_t, has_l = "timestep_bucket" in e, "layer_bucket" in e
            if not has_t and not has_l:
                if op in self._op:
                    raise ValueError("%s: a second operator-level entry" % where)
                self._op[op] = Thresholds(tau, ladder, "operator")
                continue
            tb = int(e.get("timestep_bucket", 0))
            lb = int(e.get("layer_bucket", 0))
            if not (0 <= tb < self._nbuckets(self.t_edges)) or not (0 <= lb < self._nbuckets(self.l_edges)):
                raise ValueError("%s: bucket index outside the edges" % where)
            key = (op, tb, lb)
            if key in self._bucket:
                raise ValueError("%s: a second entry for bucket %s" % (where, key))
            rows = e.get("rows")
            self._bucket[key] = (Thresholds(tau, ladder, "bucket"), None if rows is None else int(rows))

    @staticmethod
    def _nbuckets(edges) -> int:
        return 1 if edges is None else len(edges) - 1

    @staticmethod
    def _bucket_of(edges, v) -> Optional[int]:
        """Bucket of value v, or None when v lies outside the edges."""
        if edges is None:
            return 0
        if v is None or v < edges[0] or v >= edges[-1]:
            return None
        return bisect.bisect_right(edges, v) - 1

    @classmethod
    def load(cls, path: str) -> "ThresholdTable":
        with open(path) as f:
            return cls(json.load(f))

    @classmethod
    def loads(cls, text: str) -> "ThresholdTable":
        return cls(json.loads(text))

    def operators(self) -> List[str]:
        return sorted(set(self._op) | {k[0] for k in self._bucket})

    def lookup(self, operator: str, timestep: Optional[int] = None, layer: Optional[int] = None) -> Thresholds:
        """The thresholds of (operator, timestep bucket, layer bucket); the operator-level
        entry when that bucket has no entry, is sparse (fewer calibration rows than
        min_rows) or the timestep / layer lies outside the edges.  KeyError when the
        operator has neither."""
        tb = self._bucket_of(self.t_edges, timestep)
        lb = self._bucket_of(self.l_edges, layer)
        if tb is not None and lb is not None:
            hit = self._bucket.get((operator, tb, lb))
            if hit is not None:
                thr, rows = hit
                if rows is None or rows >= self.min_rows:
                    return thr
        if operator in self._op:
            return self._op[operator]
        raise KeyError("no thresholds for operator %r (bucket %s, %s) and no operator-level entry"
                       % (operator, tb, lb))


def mp_lengths_from_table(metric, table: ThresholdTable, operator: str, timestep: Optional[int] = None,
                          layer: Optional[int] = None, stream=None):
    """Per-row stream lengths on the device (``mp_lengths``) with the thresholds and ladder
    that ``table`` holds for this operator call.  Returns (L int32 tensor, Thresholds)."""
    from . import mp_lengths
    thr = table.lookup(operator, timestep, layer)
    return mp_lengths(metric, list(thr.tau), list(thr.ladder), stream=stream), thr
