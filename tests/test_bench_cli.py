"""bench.py's command line on the host: a request for more than one GPU ends before any
device work, with exit status 2 and a message that names the one-GPU limit (no GPU needed)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    for n in (2, 8):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n),
                            "--steps", "1", "--warmup", "0"],
                           cwd=ROOT, capture_output=True, text=True, timeout=120)
        assert r.returncode == 2, (r.returncode, r.stdout, r.stderr)
        assert "one GPU" in r.stderr and f"--gpus {n}" in r.stderr
        assert r.stdout.strip() == ""        # no JSON line for a run that did not happen
