"""The counter record behind the bench line's `roofline.traffic`: it is reported for the
workload and seed it was measured on, and for no other (the L2 re-fetches of the gate/up
GEMM depend on the packed plan's shape).  CPU only."""
import json

import bench


def _record():
    with open(bench.TRAFFIC_SUMMARY) as f:
        line = next(l for l in f if l.startswith("record: "))
    return json.loads(line[len("record: "):])


def test_record_states_its_workload_and_seed():
    rec = _record()
    assert rec["workload"] == "llama2-7b-lognormal" and rec["seed"] == 0
    # HBM bytes per launch = reads + writes, both already calibrated
    assert rec["hbm_bytes_per_launch"] == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]


def test_record_applies_to_its_own_workload_only():
    rec = _record()
    if rec["kernel_source_sha256"] != bench.source_sha256(bench.GEMM_SOURCE):
        assert bench.recorded_traffic("llama2-7b-lognormal", 0) is None
    else:
        assert bench.recorded_traffic("llama2-7b-lognormal", 0) == rec
    assert bench.recorded_traffic("llama-1.3b-long-zipf", 0) is None
    assert bench.recorded_traffic("llama2-7b-lognormal", 1) is None
