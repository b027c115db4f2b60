"""The boundary from plain C: include/specdec.h compiles as C99 with warnings
as errors, a C program links against libspecdec.so, and the calls that need
no GPU behave as declared (ABI version, workspace size, an argument error
with its text, and a scheduling round of the host-side SequencePool).
No kernel is launched."""
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
LIB_DIR = ROOT / "paper_2510_22876_amd"

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "specdec.h"

#define CHECK(c) do { if (!(c)) { printf("failed: %s (line %d)\n", #c, __LINE__); return 1; } } while (0)

int main(void) {
  CHECK(specdec_abi_version() == SPECDEC_ABI_VERSION);
  /* 48 logit rows of 32000: 16 workgroups of 2048 elements per row */
  CHECK(specdec_workspace_bytes(8, 5, 32000) == 256 + 8 * 6 * 16 * 8 + 16 * 8);
  /* an argument error is reported before anything is enqueued */
  CHECK(specdec_verify_greedy(NULL, SPECDEC_BF16, NULL, NULL, -1, 3, 100, 10, NULL, NULL, NULL, NULL, NULL,
                              NULL, 0, NULL, NULL) == SPECDEC_ERR_INVALID_ARGUMENT);
  CHECK(strstr(specdec_last_error(), "B=-1") != NULL);
  /* an empty batch is a no-op */
  CHECK(specdec_verify_greedy(NULL, SPECDEC_BF16, NULL, NULL, 0, 3, 100, 10, NULL, NULL, NULL, NULL, NULL,
                              NULL, 0, NULL, NULL) == SPECDEC_OK);

  /* SequencePool: four sequences, window 4, batches of 2, length-sorted */
  const int32_t lens[4] = {9, 5, 7, 5};
  specdec_sched_t* s = NULL;
  CHECK(specdec_sched_create(lens, 4, 4, 2, 100, 1, -1, &s) == SPECDEC_OK && s != NULL);
  int32_t slots[2], blens[2];
  specdec_batch_info_t info;
  CHECK(specdec_sched_next_batch(s, slots, blens, &info) == SPECDEC_OK);
  /* the two sequences of length 5 form a same-length batch */
  CHECK(info.B == 2 && info.same_length == 1 && info.width == 5 && info.reuse == 0);
  CHECK(slots[0] == 1 && slots[1] == 3 && blens[0] == 5 && blens[1] == 5);
  const int32_t n_acc[2] = {2, 2};
  CHECK(specdec_sched_commit(s, n_acc, NULL, 4) == SPECDEC_OK);
  /* every row accepted alike: the batch is kept (lazy realignment) */
  CHECK(specdec_sched_next_batch(s, slots, blens, &info) == SPECDEC_OK);
  CHECK(info.reuse == 1 && info.B == 2 && info.width == 8 && slots[0] == 1 && slots[1] == 3);
  const int32_t ragged[2] = {0, 3};
  CHECK(specdec_sched_commit(s, ragged, NULL, 4) == SPECDEC_OK);
  CHECK(specdec_sched_next_batch(s, slots, blens, &info) == SPECDEC_OK);
  CHECK(info.reuse == 0);
  int32_t all[4];
  CHECK(specdec_sched_lengths(s, all) == SPECDEC_OK);
  CHECK(all[0] == 9 && all[1] == 9 && all[2] == 7 && all[3] == 12);
  CHECK(specdec_sched_active(s) == 4);
  specdec_sched_destroy(s);
  printf("ok\n");
  return 0;
}
"""


def test_c_program_links_and_runs(tmp_path):
    if not (LIB_DIR / "libspecdec.so").exists():
        pytest.fail("libspecdec.so is not built")
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "abi"
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", f"-I{ROOT / 'include'}", str(src),
                    f"-L{LIB_DIR}", "-lspecdec", f"-Wl,-rpath,{LIB_DIR}", "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
