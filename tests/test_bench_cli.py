"""Host-side checks of the benchmark's command line (no GPU touched).

The benchmark measures one GPU: asked for more, it must refuse with a JSON
message and a non-zero status before it initialises any device.
"""
from __future__ import annotations

import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    for n in ("2", "8"):
        r = run_bench("--gpus", n, "--steps", "1", "--warmup", "0")
        assert r.returncode == 2, (n, r.returncode, r.stderr)
        line = json.loads(r.stdout.strip().splitlines()[-1])
        assert "one GPU" in line["error"]


def test_unknown_option_is_an_error():
    r = run_bench("--no-such-option")
    assert r.returncode != 0
    assert "usage" in r.stderr
