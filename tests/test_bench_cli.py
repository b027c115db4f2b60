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
    for word in ("exspec", "varlen", "chained", "verify", "--verify", "--graph", "--bound", "--noalloc", "--variant"):
        assert word in r.stdout, word


def test_traffic_comes_only_from_counters_of_the_same_step():
    """bench.py takes `roofline.traffic` from a committed counter summary only
    when the summary was taken on the current kernel sources and on a launch
    with this run's algorithmic bytes."""
    import re
    import bench
    for path in sorted((ROOT / "profiles").glob("*_hbm_counters.md")):
        text = path.read_text()
        alg = int(re.search(r"Algorithmic bytes per launch \(bench.py\):\s*(\d+)", text).group(1))
        hbm = float(re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text).group(1))
        kernel, variant, workload = path.name[:-len("_hbm_counters.md")].split("_")
        srcs = {"realign": bench.KERNEL_SRCS, "gather": bench.GATHER_SRCS, "varlen": bench.VARLEN_SRCS,
                "verifyscan": bench.KERNEL_SRCS, "samplestats": bench.SAMPLE_SRCS}[kernel]
        value, src = bench.read_traffic_summary(workload, variant, alg, kernel=kernel, srcs=srcs)
        if value is None:
            assert src == "kernel changed since the counters were taken", (path.name, src)
        else:
            assert value == hbm and src == path.name
            # the counters read the algorithmic bytes: cache moves to 0.1%; the scans to 0.5% (their algorithmic
            # bytes count the logits alone, the counters also see the partial maxima and row-boundary lines)
            tol = 5e-3 if kernel in ("verifyscan", "samplestats") else 1e-3
            assert abs(hbm / alg - 1) < tol, path.name
        value, src = bench.read_traffic_summary(workload, variant, alg + 1, kernel=kernel, srcs=srcs)
        assert value is None, path.name
    value, src = bench.read_traffic_summary("nosuch", "oop", 1)
    assert value is None and src == "no counter summary"
