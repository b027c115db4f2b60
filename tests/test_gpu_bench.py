"""bench.py's JSON line on a GPU: short runs of the default configuration
(the vicuna7b-shaped fused step) and of every other path print exactly one
line carrying every field of the benchmark contract, with a roofline of the
path's dominant kernel and the oracle's CPU baseline, and numbers that agree
with each other."""
import json
import os
import subprocess
import sys
from pathlib import Path

import pytest
import torch

from tests.gpu_util import say

pytestmark = pytest.mark.gpu

ROOT = Path(__file__).resolve().parent.parent

PATHS = [
    [],                                             # the default: vicuna7b, out of place, greedy
    ["--variant", "inplace"],
    ["--verify", "sample"],
    ["--graph"],
    ["--bound"],
    ["--bound", "--noalloc", "--variant", "inplace"],
    ["--path", "chained"],
    ["--path", "exspec"],
    ["--path", "exspec", "--exspec-batch", "same"],
    ["--path", "varlen"],
    ["--path", "verify"],
    ["--path", "verify", "--workload", "stress"],
    ["--path", "verify", "--verify", "sample"],
]


def _bench(args):
    say(f"bench.py {' '.join(args)} --steps 3 --warmup 1")
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), *args, "--steps", "3", "--warmup", "1",
                        "--cpu-baseline-seconds", "0.3", "--copy-ceiling", "0"],
                       capture_output=True, text=True, timeout=240, cwd=ROOT, env=dict(os.environ))
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


@pytest.mark.parametrize("args", PATHS, ids=lambda a: "-".join(x.lstrip("-") for x in a) or "default")
def test_bench_line(args):
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    d = _bench(args)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    unit = "calls/s" if "verify" in args and "--path" in args else "steps/s"
    assert d["unit"] == unit and d["higher_is_better"] is True and d["dtype"] == "bf16"
    assert d["value"] > 0 and abs(d["value"] * d["ms_per_step"] - 1e3) < 1e-3
    assert "workload" in d["config"]
    if not args:
        assert "vicuna7b" in d["config"]["workload"] and "out-of-place" in d["config"]["workload"]
    rf = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in rf, key
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert 0 < rf["achieved"] < rf["peak"] and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    cb = d["cpu_baseline"]
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in cb, key
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0
