"""The HBM counter records that bench.py reports as ``roofline.traffic``
exist for every workload and are well formed (for the copies, one figure
per launch kind the counters saw), and every profile summary
names the command that made it.  (bench.py reports a record only while the
kernel sources hash to the value stored in it, and null traffic otherwise.)"""
import json
import os

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
WORKLOADS = ["handoff", "relayout", "mla", "host_tier", "tp_reshard", "cow_fork",
             "handoff_layered", "small_requests", "host_tier_v", "page_hash"]


@pytest.mark.parametrize("name", WORKLOADS)
def test_traffic_record_is_well_formed(name):
    path = os.path.join(ROOT, "profiles", f"traffic_{name}.json")
    assert os.path.exists(path), f"profiles/traffic_{name}.json missing"
    rec = json.load(open(path))
    assert rec["traffic_bytes_per_launch"] > 0
    assert rec["fetch_scale"] > 0 and rec["write_scale"] > 0
    if name != "page_hash":
        # per launch kind of the roofline's kernel: bench.py reports the one its timed steps took
        assert rec["by_launch"] and set(rec["by_launch"]) <= {"sweep", "grid"}
        assert all(v > 0 for v in rec["by_launch"].values())
        assert rec["traffic_bytes_per_launch"] in rec["by_launch"].values()
    assert len(rec["kernel_sha"]) == 16
    # reported only while the sources match the ones the counters were taken on
    assert (bench.traffic_record(name) is not None) == (rec["kernel_sha"] == bench.kernel_sha(name))


def test_profile_summaries_name_their_command():
    for fn in os.listdir(os.path.join(ROOT, "profiles")):
        if fn.endswith(".md"):
            text = open(os.path.join(ROOT, "profiles", fn)).read()
            assert "rocprofv3" in text and "bench.py" in text, fn
        elif fn.endswith(".json"):
            json.load(open(os.path.join(ROOT, "profiles", fn)))
