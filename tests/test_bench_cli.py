"""bench.py's command line on the CPU: more than one GPU is refused with a message and a
non-zero status before anything touches a device."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    for n in (2, 8):
        p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)], capture_output=True,
                           text=True, timeout=300, cwd=ROOT)
        assert p.returncode != 0
        rec = json.loads(p.stdout.strip().splitlines()[-1])
        assert rec["n_gpus_requested"] == n and "one GPU" in rec["error"]
