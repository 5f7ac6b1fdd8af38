"""The threshold table of the per-row length policy (Sec. 4.4, "Threshold fitting"): lookup by
operator, timestep bucket and layer bucket, operator-level fallback, validation (CPU)."""
import json
import os

import numpy as np
import pytest

from paper_2609_32922_amd.thresholds import ThresholdTable

HERE = os.path.dirname(os.path.abspath(__file__))
FIXTURE = os.path.join(HERE, "golden", "thresholds_synthetic.json")


@pytest.fixture(scope="module")
def table():
    return ThresholdTable.load(FIXTURE)


def test_bucket_hit_and_edges(table):
    t = table.lookup("mlp_fc1", timestep=3, layer=27)          # bucket (0, 3)
    assert t.source == "bucket" and t.tau == (0.6, 0.3, 0.1) and t.ladder == (192, 96, 48, 24)
    # bucket edges are half-open: timestep 10 is bucket 1, layer 21 is bucket 3
    assert table.lookup("mlp_fc2", timestep=10, layer=21).source == "bucket"
    assert table.lookup("mlp_fc2", timestep=9, layer=21).source == "operator"
    # an entry's own ladder overrides the default
    assert table.lookup("mlp_fc2", timestep=24, layer=27).ladder == (256, 128, 64, 32)


def test_operator_level_fallback(table):
    # no entry for the bucket
    t = table.lookup("mlp_fc1", timestep=30, layer=5)
    assert t.source == "operator" and t.tau == (0.75, 0.5, 0.25)
    # a sparse bucket (100 calibration rows < min_rows 256) falls back
    assert table.lookup("mlp_fc1", timestep=40, layer=0).source == "operator"
    # outside the edges (and no timestep at all) falls back
    assert table.lookup("mlp_fc1", timestep=50, layer=0).source == "operator"
    assert table.lookup("mlp_fc1", timestep=None, layer=27).source == "operator"
    assert table.lookup("mlp_fc1", timestep=3, layer=-1).source == "operator"
    # an operator with bucket entries only has no fallback
    assert table.lookup("qk", timestep=0, layer=0).source == "bucket"
    with pytest.raises(KeyError):
        table.lookup("qk", timestep=30, layer=0)
    with pytest.raises(KeyError):
        table.lookup("unknown_op", timestep=0, layer=0)
    # one level: no thresholds
    assert table.lookup("proj").ladder == (64,) and table.lookup("proj").tau == ()
    assert table.operators() == ["av", "mlp_fc1", "mlp_fc2", "proj", "qk"]


def test_models_without_timesteps():
    t = ThresholdTable.loads(json.dumps({
        "ladder": [128, 64], "layer_edges": [0, 12],
        "entries": [{"operator": "qk", "layer_bucket": 0, "tau": [0.5]},
                    {"operator": "qk", "tau": [0.9]}]}))
    assert t.lookup("qk", layer=3).tau == (0.5,)          # any timestep, one bucket
    assert t.lookup("qk", timestep=7, layer=3).tau == (0.5,)
    assert t.lookup("qk", layer=12).tau == (0.9,)


@pytest.mark.parametrize("entry,msg", [
    ({"operator": "x", "tau": [0.2, 0.5]}, "not increase"),
    ({"operator": "x", "tau": [1.5, 0.5]}, "not increase"),
    ({"operator": "x", "tau": [0.5]}, "thresholds for"),
    ({"operator": "x", "tau": [0.5, 0.4], "ladder": [64, 64, 32]}, "strictly decreasing"),
    ({"operator": "x", "tau": [0.5, 0.4], "ladder": [8192, 64, 32]}, "integers in"),
    ({"operator": "x", "tau": [0.5, 0.4], "timestep_bucket": 5}, "outside the edges"),
])
def test_rejects_bad_entries(entry, msg):
    doc = {"ladder": [96, 48, 24], "timestep_edges": [0, 10, 20], "entries": [entry]}
    with pytest.raises(ValueError, match=msg):
        ThresholdTable(doc)
    with pytest.raises(ValueError, match="a second"):
        ThresholdTable({"ladder": [96, 48, 24], "entries": [{"operator": "x", "tau": [0.5, 0.4]}] * 2})


def test_table_thresholds_drive_the_policy(table, oracle_mod):
    # the looked-up thresholds and ladder, through the oracle's definition of the policy:
    # rows at or above tau_1 of the normalised metric get L_1, rows below every threshold
    # the shortest level
    thr = table.lookup("mlp_fc1", timestep=3, layer=27)
    g = np.linspace(0.0, 1.0, 101).astype(np.float32)
    L = oracle_mod.mp_lengths_fp32(g, thr.tau, thr.ladder)
    assert set(L.tolist()) == set(thr.ladder)
    assert np.all(L[g >= 0.6] == 192) and np.all(L[g < 0.1] == 24)
    assert np.all(np.diff(L) >= 0)       # longer streams for larger metrics
