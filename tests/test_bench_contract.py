"""bench.py contract checks that need no GPU: one GPU only, and the counted scan
traffic it reports is tied to the scan sources it was measured on."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_scan_traffic_is_reported_only_for_the_measured_sources():
    import bench
    for w, entry in bench.SCAN_TRAFFIC.items():
        assert w in bench.WORKLOADS
        assert os.path.exists(os.path.join(ROOT, entry[-1])), entry[-1]
        traffic, detail = bench.scan_traffic(w)
        if entry[0] == bench.scan_sources_sha():
            assert traffic > 0 and abs(traffic - detail["fetch_bytes"] - detail["write_bytes"]) <= 1
        else:
            assert traffic is None and detail is None
    assert bench.scan_traffic("no-such-workload") == (None, None)
