"""bench.py's command-line contract, checked without a GPU."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_unit_bytes_accounting():
    sys.path.insert(0, ROOT)
    import bench
    n, K, R = 1000, 8, 2
    p1, p2 = bench.unit_bytes(n, K, R, active=8, rolled_back=False)
    assert p1 == n * (4 + K * R) and p2 == n * (8 + K * R + 8 + K * R)  # 20 + 48 B per element
    _, p2_masked = bench.unit_bytes(n, K, R, active=6, rolled_back=False)
    assert p2 - p2_masked == n * 2 * R  # flagged workers' replicas are not read
    _, p2_rb = bench.unit_bytes(n, K, R, active=0, rolled_back=True)
    assert p2_rb == n * (4 + K * R)  # rollback: read theta, write the replicas
    assert bench.unit_bytes(n, K, R, 8, False, one_pass=True) == (n * (16 + 2 * K * R), 0)
