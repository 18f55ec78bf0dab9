"""Host-side parts of the benchmark's contract (no GPU): more than one GPU
is refused with a message and exit status 2 before anything touches a GPU,
and a stored HBM-traffic figure is only reported for the workload, schedule
and kernel source it was measured on."""

import hashlib
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "ONE GPU" in msg["error"]


def test_traffic_figures_follow_the_measured_source():
    for (kernel, mode), m in bench.MEASURED_TRAFFIC.items():
        path = os.path.join(ROOT, "paper_2609_07108_amd", "csrc", m["source"])
        current = hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]
        got = bench.measured_traffic(kernel, "eagle3-K3-L262144-cp8r0", mode)
        assert got == (m["bytes"] if current == m["sha256_16"] else None)
        # never for another workload or an unmeasured schedule
        assert bench.measured_traffic(kernel, "dflash16-L32768", mode) is None
        assert bench.measured_traffic(kernel, "eagle3-K3-L262144-cp8r0", "no-such-mode") is None
