"""The ablation harness end to end on a small topic-structured case: every
configuration runs through the library, density 100 % covers all the mass,
and no selection covers more mass than the best-by-mass one of its size."""
import argparse

import pytest
import torch

import bench

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("data", ["topics", "planted"])
def test_ablation_runs_and_is_bounded(data):
    args = argparse.Namespace(ablation_tokens=4096, ablation_layers=2, ablation_needles=6,
                              ablation_data=data, ablation_drift=0.1)
    out = bench.run_ablation(args, torch.device("cuda:0"))
    rows = out["rows"]
    best = {r["value"]: r["mass_recall"] for r in rows if r["axis"] == "best"}
    for r in rows:
        if r["axis"] == "best":
            continue
        assert 0.0 < r["mass_recall"] <= best[r["pct"]] + 1e-9, r
        if r["pct"] == 100:
            assert r["mass_recall"] == pytest.approx(1.0, abs=1e-9)
            assert r["selected_fraction"] == pytest.approx(1.0)
        if data == "planted":
            assert r["needle_recall"] is not None
