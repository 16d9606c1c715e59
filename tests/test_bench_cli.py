"""bench.py's command-line contract, checked without a GPU: more than one
GPU is refused with a message (the path runs on one GPU), so is a token
count outside the fp4 stack's range, and the traffic record it reads from
profiles/ parses."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_batch_only_range_is_checked():
    for b in ("1", "17"):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--batch-only", b],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode == 2
        assert "2..16" in r.stderr
        assert r.stdout == ""


def test_traffic_record_parses_or_is_null():
    sys.path.insert(0, ROOT)
    import bench
    t = bench.traffic_record()
    assert t is None or t > 1e9     # bytes per launch of the 1.6 GB stack
