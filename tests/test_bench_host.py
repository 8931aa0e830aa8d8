"""Host-side parts of bench.py's contract that need no GPU: more than one GPU
is refused with a message, unknown workloads are rejected, and the committed
counter summary parses into the roofline's traffic figure."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_unknown_workload_is_rejected():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "nope"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "invalid choice" in r.stderr


def test_committed_counters_parse():
    b = _bench()
    txt = open(b.COUNTER_FILE).read()
    assert "kernel_source_digest:" in txt and "hbm_bytes_per_launch:" in txt
    t = b.committed_traffic()
    # null only when the row kernel's sources changed after the counters were taken
    if t is not None:
        alg = 39320 * 3 * 151936 * 2 + (65536 - 39320) * 151936 * 2
        assert 1.0 <= t / alg < 1.05
    assert len(b.row_kernel_digest()) == 16
