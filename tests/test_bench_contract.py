"""bench.py reports stored HBM counters only for the kernel and workload they were taken on."""
import json

import bench

KEY = {"config": "q235b", "seed": 3, "gate_policy": "topb", "page_size": 0, "serve": False}


def test_traffic_only_for_the_profiled_kernel_and_workload(tmp_path):
    h = "ab" * 32
    path = tmp_path / "pmc.json"
    path.write_text(json.dumps({"attn_src_sha256": h, "workload_key": KEY,
                                "hbm_bytes_per_launch": 1.25e9}))
    assert bench.traffic_from_profile(h, dict(KEY), str(path)) == 1.25e9
    for change in ({"config": "l8b"}, {"seed": 4}, {"gate_policy": "sparse"},
                   {"page_size": 64}, {"serve": True}):
        assert bench.traffic_from_profile(h, {**KEY, **change}, str(path)) is None
    assert bench.traffic_from_profile("cd" * 32, dict(KEY), str(path)) is None
    assert bench.traffic_from_profile(h, dict(KEY), str(tmp_path / "absent.json")) is None


def test_committed_summary_names_its_workload():
    with open(bench.PMC_SUMMARY) as f:
        d = json.load(f)
    assert d["workload_key"] == KEY
    assert len(d["attn_src_sha256"]) == 64 and d["hbm_bytes_per_launch"] > 0
