"""bench.py's command line on the host: it measures one GPU and refuses more."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert p.returncode == 2
    assert "one GPU only" in p.stderr and p.stdout == ""


def test_bench_rejects_unknown_workload():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "no_such_workload"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert p.returncode != 0 and "invalid choice" in p.stderr
