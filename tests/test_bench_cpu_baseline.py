"""bench.py's cpu_baseline: the oracle timed on a stratified sample, through one layer and
then through as many further layers as its time budget allows, never more than the model
has.  CPU only (the tiny workload's shape, 3 layers)."""
import re

import pytest

import bench
from paper_2404_09529_amd import workloads as W


@pytest.mark.parametrize("budget_s,layers_run", [(0.0, 1), (1e9, 3)])
def test_layers_timed_follow_the_budget(monkeypatch, budget_s, layers_run):
    monkeypatch.setattr(bench, "CPU_SAMPLE_S", budget_s)
    case = W.make_case(1, 0, n_layers=3)
    r = bench.cpu_baseline(case)
    m = re.search(r"each through (\d+) of the (\d+) layers", r["sample"])
    assert m and (int(m.group(1)), int(m.group(2))) == (layers_run, 3), r["sample"]
    assert r["value"] > 0 and r["kind"] == "oracle" and r["dtype"] == "f32"
