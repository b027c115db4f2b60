"""Host-sanitizer builds for CPU-only checks.

Builds, out of tree under ``paper_2510_22876_amd/_build/hostsan/``:

* the library with its host code (argument validation, the scheduler, launch
  set-up) instrumented by AddressSanitizer and UndefinedBehaviorSanitizer;
  device code is compiled as usual (the sanitizer flags apply to the host
  pass only);
* the CPU oracle, instrumented the same way (clang, matching the runtime).

Usage: ``python -m paper_2510_22876_amd.build_hostsan`` prints the command
that runs the CPU tests against both builds with clang's sanitizer runtime
preloaded (``SPECDEC_LIB`` and ``SPECDEC_ORACLE_LIB`` select the builds).
The mutation tests compile their own oracles and are left out of that run.
Not for GPU runs: the instrumented host code is for CPU checks only.
"""
from __future__ import annotations

import glob
import subprocess
from pathlib import Path

from paper_2510_22876_amd import build as hip_build

OUT = hip_build.PKG / "_build" / "hostsan"
HOST_SAN = ["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]


def build() -> tuple[Path, Path]:
    OUT.mkdir(parents=True, exist_ok=True)
    common = list(hip_build.COMMON)
    try:
        hip_build.COMMON[:] = common + HOST_SAN
        lib = hip_build.build(out=OUT / "libspecdec.so", build_dir=OUT / "obj")
    finally:
        hip_build.COMMON[:] = common
    oracle_lib = OUT / "libspecdec_oracle.so"
    subprocess.run(["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                    "-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=undefined",
                    str(hip_build.ROOT / "oracle" / "specdec_oracle.c"), "-o", str(oracle_lib), "-lm"], check=True)
    return lib, oracle_lib


def runtime() -> str:
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise FileNotFoundError("clang's AddressSanitizer runtime not found under /opt/rocm/llvm")
    return found[-1]


if __name__ == "__main__":
    lib, oracle_lib = build()
    print(f"SPECDEC_LIB={lib} SPECDEC_ORACLE_LIB={oracle_lib} LD_PRELOAD={runtime()} "
          "ASAN_OPTIONS=detect_leaks=0:halt_on_error=1 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 "
          "python -m pytest tests -x -q -m 'not gpu' -p no:cacheprovider --deselect tests/test_oracle_mutants.py")
