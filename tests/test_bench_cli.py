"""The bench contract on the host: more than one GPU is refused with a
message (the path runs on one device), and the algorithmic byte counts
follow their per-record and per-row definitions."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes_definition():
    sys.path.insert(0, ROOT)
    import bench
    n, nm, rows, depth, nc = 1000, 300, 400, 4, 16
    b = bench.algorithmic_bytes(n, nm, rows, depth, nc, 200)
    # each part grows with its own count
    assert bench.algorithmic_bytes(n + 1, nm, rows, depth, nc, 200) - b == \
        19 + 8 * nc + 40 + 4 * depth
    assert bench.algorithmic_bytes(n, nm, rows + 1, depth, nc, 200) - b == \
        4 * depth + 1 + 1 + 8 + 5 * 8 + 4 + 8 * nc + 6 * 8
