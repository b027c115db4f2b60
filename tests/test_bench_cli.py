"""bench.py's command-line contract on the host: more than one GPU (by flag
or by a torchrun world size) is refused with a message, before any device
work; the help text lists every path."""
import os
import subprocess
import sys
from pathlib import Path

ROOT = Path(__file__).resolve().parent.parent


def _run(*args, env=None):
    return subprocess.run([sys.executable, str(ROOT / "bench.py"), *args], capture_output=True, text=True,
                          env={**os.environ, **(env or {})}, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""
    r = _run(env={"WORLD_SIZE": "4"})
    assert r.returncode == 2 and "WORLD_SIZE=4" in r.stderr and r.stdout == ""


def test_help_lists_the_paths():
    r = _run("--help")
    assert r.returncode == 0
    for word in ("exspec", "varlen", "chained", "--verify", "--graph", "--variant"):
        assert word in r.stdout, word
