"""Pins the oracle's accounting against the numbers the paper prints.

Section 4.1 "Metrics" defines Hit = 1 - D/A, AdjHit = (A - D)/(A + P) and
Load/token = (D + P) S_exp / T.  Every decode token accesses K experts at each
of L layers, so A = T L K.  Tables 1 and 3 then fix D and P from the printed
Hit and AdjHit, and the printed Load must follow with S_exp the bytes of one
whole bf16 SwiGLU expert (3 d F x 2 bytes) in decimal MB.  A wrong unit (MiB,
fp32 experts, per-layer T) or a wrong formula misses by far more than the
0.1% tolerance.
"""
import json
import os

import pytest

import oracle
from synth import WORKLOADS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_metrics.json")
DOC = json.load(open(GOLDEN))


def _ids(rows):
    return [f"{r['method']}-{r['model']}-{r['task']}-{r.get('capacity', '')}-{r.get('R', '')}" for r in rows]


@pytest.mark.parametrize("row", DOC["rows"], ids=_ids(DOC["rows"]))
def test_printed_rows_satisfy_metric_definitions(row):
    m = DOC["models"][row["model"]]
    T = 1_000_000
    A = T * m["L"] * m["K"]
    hit = row["hit"] / 100.0
    D = round(A * (1.0 - hit))
    if row["adj_hit"] is None:          # update-only: P = 0, AdjHit = Hit
        P = 0
    else:
        P = round(A * hit / (row["adj_hit"] / 100.0) - A)
    s_exp = 3 * m["d"] * m["F"] * 2
    h, adj, load = oracle.metrics(A, D, P, T, s_exp)
    assert abs(h * 100 - row["hit"]) < 1e-4
    if row["adj_hit"] is None:
        assert abs(h - adj) < 1e-12          # AdjHit equals Hit when P = 0
    else:
        assert abs(adj * 100 - row["adj_hit"]) < 1e-4
    tol = row.get("rel_tol", DOC["default_rel_tol"])
    assert abs(load - row["load_mb"]) <= tol * row["load_mb"], (load, row["load_mb"])


def test_known_outlier_rows_really_deviate():
    # The two GPT-OSS Spatio-Temporal rows are recorded with a wider tolerance;
    # make sure that wider tolerance is not hiding a unit error everywhere.
    outliers = [r for r in DOC["rows"] if "rel_tol" in r]
    assert len(outliers) == 2
    assert all(r["model"] == "gptoss" and r["method"] == "Spatio-Temporal Router" for r in outliers)


@pytest.mark.parametrize("p", DOC["added_params"], ids=lambda p: f"{p['model']}-{p['routers']}")
def test_added_router_parameters_pin_router_shape(p):
    # each auxiliary router is a bias-free d -> N map per layer
    w = WORKLOADS["qwen3_30b"] if p["model"] == "qwen3" else WORKLOADS["gptoss_20b"]
    n = p["routers"] * w.L * w.N * w.d
    assert abs(n - p["params"]) <= 0.01 * p["params"]


def test_expert_bytes_of_workloads():
    assert WORKLOADS["qwen3_30b"].expert_bytes == 9_437_184
    assert WORKLOADS["gptoss_20b"].expert_bytes == 49_766_400
    assert WORKLOADS["qwen3_235b_slice"].expert_bytes == 37_748_736
