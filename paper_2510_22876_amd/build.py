"""Build libspecdec.so for gfx950 with hipcc (in-tree, next to this file).

Usage: ``python -m paper_2510_22876_amd.build``.  Every HIP source is compiled
with packed-FP32 instructions disabled (``-packed-fp32-ops``).
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
LIB = PKG / "libspecdec.so"
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          f"-I{ROOT / 'include'}", f"-I{CSRC}"]


def build(verbose: bool = False, defines=(), out: Path = LIB, build_dir: Path | None = None) -> Path:
    """Compile every source under csrc/ and link ``out``.  ``defines`` adds
    -D options (the kernels' compile-time tunables)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    objs = []
    out_dir = build_dir or (PKG / "_build")
    out_dir.mkdir(parents=True, exist_ok=True)
    extra = [f"-D{d}" for d in defines]
    for src in sorted(CSRC.glob("*.hip")) + sorted(CSRC.glob("*.cpp")):
        obj = out_dir / (src.name + ".o")
        cmd = [hipcc, *COMMON, *extra, "-c", str(src), "-o", str(obj)]
        if src.suffix == ".cpp":
            cmd = [hipcc, *COMMON, *extra, "-x", "hip", "-c", str(src), "-o", str(obj)]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        objs.append(str(obj))
    tmp = Path(out).with_suffix(".so.tmp")
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", str(tmp)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return Path(out)


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
