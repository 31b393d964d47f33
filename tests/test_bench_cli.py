"""bench.py's command line on the CPU: a request for more than one GPU is refused with a message,
before any device work (the step is measured on one GPU)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "GPU" in (r.stdout + r.stderr)


def test_committed_traffic_matches_the_current_predictor_source():
    # the bench line's roofline.traffic is reported only for the kernel source the counters
    # were taken on; the committed record must be for the current source and workload
    sys.path.insert(0, ROOT)
    import bench
    import json
    rec = json.load(open(bench.TRAFFIC_FILE))
    for name in ("c4", "c3"):   # the headline workload and the chained one
        t = bench.measured_traffic(name)
        assert t is not None, "profiles/predict_traffic.json was taken on another predictor source"
        r = rec["records"][name]
        assert t == r["hbm_bytes_per_launch"] >= r["algorithmic_bytes_per_launch"] > 0
    assert bench.measured_traffic("c1") is None
