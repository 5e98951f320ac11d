"""Host-side checks of the benchmark's contract: one GPU only, and the HBM-traffic record is
reported only for the kernel source it was measured on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode != 0
    assert "--gpus 1" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line


def test_traffic_record_is_consistent_and_tied_to_its_source():
    sys.path.insert(0, ROOT)
    import bench
    import hashlib
    text = open(bench.TRAFFIC_SUMMARY).read()
    body = json.loads(text.split("```json\n")[1].split("\n```")[0])
    for key in ("rope_off", "rope_on"):
        e = body[key]
        assert e["hbm_bytes_per_launch"] == e["read_bytes"] + e["write_bytes"]
        assert e["read_bytes"] == round(e["fetch_size_kib_raw"] * body["fetch_scale"] * 1024)
        assert e["write_bytes"] == round(e["write_size_kib_raw"] * body["write_scale"] * 1024)
        assert abs(e["traffic_over_algorithmic"] - e["hbm_bytes_per_launch"] / e["algorithmic_bytes"]) < 1e-3
    wl, pps = body["workload"], body["rope_off"]["pages_per_split"]
    current = hashlib.sha256(open(bench.KERNEL_SOURCE, "rb").read()).hexdigest() == body["decode_hip_sha256"]
    got = bench.counter_traffic(False, wl, pps)
    # reported exactly while the record belongs to this source, never otherwise
    assert got == (body["rope_off"]["hbm_bytes_per_launch"] if current else None)
    assert bench.counter_traffic(False, "some-other-workload", pps) is None
    assert bench.counter_traffic(False, wl, pps + 1) is None
