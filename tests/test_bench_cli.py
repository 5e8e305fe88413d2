"""The benchmark's command line without a GPU: a multi-GPU request is refused
with a message (the path shards by world, but only one GPU is driven), and
--aa without --rgb is an argument error."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    p = _run("--gpus", "2", "--steps", "1", "--warmup", "0")
    assert p.returncode == 2
    msg = json.loads(p.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_aa_needs_rgb():
    p = _run("--aa")
    assert p.returncode == 2
    assert "--aa needs --rgb" in p.stderr
