"""Host logic of bench.py: which committed traffic record a bench line may use."""
import json
import os

import bench


def test_traffic_keys_separate_the_launch_shapes():
    base = bench.traffic_key("l32_32k", 1024, 64, False)
    keys = {base,
            bench.traffic_key("l32_32k", 1024, 64, True),
            bench.traffic_key("l32_32k", 1024, 32, False),
            bench.traffic_key("l32_32k", 1024, 64, False, shared_layers=3),
            bench.traffic_key("l32_32k", 1024, 64, False, schedule=1),
            bench.traffic_key("l32_32k", 1024, 64, False, schedule=2)}
    assert len(keys) == 6
    assert base == "l32_32k_b1024_w64"  # the default line's record keeps its key


def test_recorded_traffic_only_for_recorded_shapes():
    path = os.path.join(bench.ROOT, "profiles", "traffic.json")
    recorded = set(json.load(open(path)))
    # shared-index mode sweeps 3 layers: it must not pick up the 32-layer record
    assert bench.traffic_key("l32_32k", 1024, 64, False, shared_layers=3) not in recorded
    assert bench.recorded_traffic(bench.traffic_key("l32_32k", 1024, 64, False,
                                                    shared_layers=3)) is None
    for key in recorded:
        rec = json.load(open(path))[key]
        assert rec["hbm_bytes_per_launch"] == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
