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


def test_roof_kernel_bytes_per_path():
    """The records reduction's bytes: fast path (two finest levels' rows,
    records in input order or through korder) and general path (gathered
    items in place of gpu, class and path)."""
    import bench
    n, depth, nc, rows = 1000, 4, 16, 300
    per_row = 4 * depth + 1 + 1 + 4 + 8 * (6 + nc)
    fast = bench.roof_kernel_bytes("agg_fast_reduce_records", n, depth, nc,
                                   rows, True)
    assert fast == n * (2 + 4 * depth + 32 + 8 * nc) + rows * per_row
    assert bench.roof_kernel_bytes("agg_fast_reduce_records", n, depth, nc,
                                   rows, False) == fast + 4 * n
    gen = bench.roof_kernel_bytes("agg_reduce_records", n, depth, nc, rows,
                                  False)
    assert gen == n * (6 + 4 * depth + 32 + 8 * nc) + rows * per_row
