"""The HBM counter records that bench.py reports as ``roofline.traffic``
exist for every workload and were taken on the kernel sources as they
stand, and every profile summary names the command that made it."""
import json
import os

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
WORKLOADS = ["handoff", "relayout", "mla", "host_tier", "tp_reshard", "cow_fork",
             "handoff_layered", "small_requests", "host_tier_v", "page_hash"]


@pytest.mark.parametrize("name", WORKLOADS)
def test_traffic_record_is_current(name):
    rec = bench.traffic_record(name)
    assert rec is not None, f"profiles/traffic_{name}.json missing or taken on other sources"
    assert rec["traffic_bytes_per_launch"] > 0
    assert rec["fetch_scale"] > 0 and rec["write_scale"] > 0


def test_profile_summaries_name_their_command():
    for fn in os.listdir(os.path.join(ROOT, "profiles")):
        if fn.endswith(".md"):
            text = open(os.path.join(ROOT, "profiles", fn)).read()
            assert "rocprofv3" in text and "bench.py" in text, fn
        elif fn.endswith(".json"):
            json.load(open(os.path.join(ROOT, "profiles", fn)))
