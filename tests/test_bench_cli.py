"""bench.py's argument checks that end the run before any GPU work: more
than one GPU, and a batch size out of range, each exit with status 2 and one
JSON line that says why (CPU only)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=300, cwd=ROOT)
    return r.returncode, r.stdout.strip().splitlines()


def test_more_than_one_gpu_is_refused():
    rc, out = _run("--gpus", "2")
    assert rc == 2
    msg = json.loads(out[-1])["error"]
    assert "one GPU" in msg


@pytest.mark.parametrize("b", ["0", "65536"])
def test_batch_out_of_range_is_refused(b):
    rc, out = _run("--batch", b)
    assert rc == 2
    assert "--batch" in json.loads(out[-1])["error"]
