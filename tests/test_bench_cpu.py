"""bench.py host logic on the CPU: the one-GPU contract and the stored traffic
figure (reported only for the kernel sources and schedule it was taken on)."""
import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_stored_traffic_follows_sources_and_schedule():
    import bench
    txt = open(os.path.join(ROOT, bench.TRAFFIC_PROFILE)).read()
    recorded = re.search(r"^kernel source hash:\s*([0-9a-f]+)", txt, re.M).group(1)
    sched = re.search(r"^schedule:\s*(\w+)", txt, re.M).group(1)
    val = bench.stored_traffic(sched)
    if recorded == bench.kernel_source_hash():
        assert val is not None and val > 6.144e6  # at least the algorithmic bytes of one call
    else:
        assert val is None  # counters of other sources are not reported
    other = "staged" if sched != "staged" else "inline"
    assert bench.stored_traffic(other) is None
