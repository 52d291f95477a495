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


def test_algorithmic_bytes_and_flops_by_hand():
    """The roofline's byte and FLOP counts on a two-request batch worked out by hand:
    request 0 has a 3-key prefix and slots {root, child}, request 1 a 5-key prefix and
    only its root; Hq = 4, Hkv = 2, D = 128."""
    import numpy as np

    class Cfg:
        head_dim, hq, hkv, R = 128, 4, 2, 2

    batch = {"prefix_len": np.array([3, 5], np.int32)}
    # slot 0: root of request 0 (sees itself), slot 1: its child (root + itself),
    # slot 2: root of request 1
    mask = np.array([[0b01], [0b11], [0b01]], np.uint32)
    res = {"q_offsets": np.array([0, 2, 3], np.int32), "tree_mask": mask}
    nbytes, flops = bench.attn_algorithmic(batch, res, Cfg)
    D, hq, hkv, nq = 128, 4, 2, 3
    kv = 4 * hkv * D * (3 + 5)                                   # prefix K and V, bf16
    rows = nq * (2 * hq * D + 4 * hkv * D + 4 * hq * D + 4 * hq)  # q, new k/v, out, lse
    assert nbytes == kv + rows
    keys = (3 + 1) + (3 + 2) + (5 + 1)                           # visible keys per slot
    assert flops == 4 * D * hq * keys
