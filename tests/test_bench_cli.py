"""bench.py's command-line contract that holds without a GPU: one GPU only (any other
count exits with status 2 and says why), and the kernel-source digest that keys the
committed counter summaries."""

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    for n in ("2", "8"):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", n],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 2
        assert "one GPU" in r.stderr
        assert r.stdout == ""


def test_counter_summaries_are_keyed_to_the_device_code():
    sys.path.insert(0, ROOT)
    import bench

    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
        summary = json.load(f)
    # a summary taken on other device code reports no traffic
    if summary["source_hash"] != h:
        assert bench.measured_traffic("kimi_headline/refresh") is None
    else:
        assert bench.measured_traffic("kimi_headline/refresh") > 0
