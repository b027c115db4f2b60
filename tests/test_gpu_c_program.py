"""The fused step driven from a plain C program: device memory from the HIP
runtime (hipMalloc / hipMemcpy), no PyTorch in the process, the library
called through include/specdec.h only.  The program reads seeded inputs from
a file, runs specdec_step (with the token row, out of place or in place) on the null
stream, and writes every output back; the outputs must equal the oracle's
element by element, and out of place the columns the step does not own keep
the sentinels the program wrote there.  In place the cache and the token row
are updated in their own buffers."""
import shutil
import subprocess
from pathlib import Path

import numpy as np
import pytest
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests.gpu_util import PAD_ID, say

pytestmark = pytest.mark.gpu

ROOT = Path(__file__).resolve().parent.parent
LIB_DIR = ROOT / "paper_2510_22876_amd"

PROGRAM = r"""
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <hip/hip_runtime_api.h>
#include "specdec.h"

static void* read_n(FILE* f, size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p || (n && fread(p, 1, n, f) != n)) { fprintf(stderr, "short input\n"); exit(3); }
  return p;
}

/* device buffer of n bytes, filled from host memory (or with byte `fill`) */
static void* dev(const void* host, size_t n, int fill) {
  void* d = NULL;
  if (hipMalloc(&d, n ? n : 16) != hipSuccess) { fprintf(stderr, "hipMalloc failed\n"); exit(4); }
  if (host && hipMemcpy(d, host, n, hipMemcpyHostToDevice) != hipSuccess) exit(5);
  if (!host && hipMemset(d, fill, n ? n : 16) != hipSuccess) exit(5);
  return d;
}

static void write_back(FILE* f, const void* d, size_t n) {
  void* h = malloc(n ? n : 1);
  if (!h || hipMemcpy(h, d, n, hipMemcpyDeviceToHost) != hipSuccess) exit(6);
  fwrite(h, 1, n, f);
  free(h);
}

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  int32_t h[13];
  if (fread(h, sizeof(int32_t), 13, in) != 13) return 3;
  const int in_place = h[12];
  const int32_t B = h[0], k = h[1], V = h[2], W_in = h[3], L = h[4], H = h[5], D = h[6], cap = h[7];
  const int32_t pm_cap = h[8], s_in_stride = h[9], s_out_stride = h[10], pad_id = h[11];
  const size_t n_logits = (size_t)B * (k + 1) * V * 2, n_draft = (size_t)B * k * 4, n_b = (size_t)B * 4;
  const size_t n_kv = (size_t)L * 2 * B * H * cap * D * 2;
  const size_t n_s_in = (size_t)B * s_in_stride * 4, n_s_out = (size_t)B * s_out_stride * 4;
  void* logits = read_n(in, n_logits);
  void* draft = read_n(in, n_draft);
  void* pad_in = read_n(in, n_b);
  void* kv = read_n(in, n_kv);
  void* s_in = read_n(in, n_s_in);
  fclose(in);

  void* d_logits = dev(logits, n_logits, 0);
  void* d_draft = dev(draft, n_draft, 0);
  void* d_pad_in = dev(pad_in, n_b, 0);
  void* d_src = dev(kv, n_kv, 0);
  void* d_dst = in_place ? d_src : dev(NULL, n_kv, 0x7F);   /* sentinel bytes outside the new width */
  void* d_s_in = dev(s_in, n_s_in, 0);
  void* d_s_out = in_place ? d_s_in : dev(NULL, n_s_out, 0x55);
  void* d_tokens = dev(NULL, (size_t)B * (k + 1) * 4, 0);
  void* d_n_acc = dev(NULL, n_b, 0);
  void* d_bonus = dev(NULL, n_b, 0);
  void* d_pad_out = dev(NULL, n_b, 0);
  void* d_w_new = dev(NULL, 4, 0);
  void* d_pos = dev(NULL, (size_t)B * pm_cap * 8, 0x66);
  void* d_mask = dev(NULL, (size_t)B * pm_cap, 0x77);
  void* d_status = dev(NULL, 4, 0);
  const size_t ws_bytes = specdec_workspace_bytes(B, k, V);
  void* d_ws = dev(NULL, ws_bytes, 0x33);    /* the workspace needs no initialisation */

  specdec_kv_t src = {d_src, L, B, H, D, cap};
  specdec_kv_t dst = {d_dst, L, B, H, D, cap};
  int32_t w_host = -1;
  const specdec_status_t st = specdec_step(d_logits, SPECDEC_BF16, (const int32_t*)d_draft, (const int32_t*)d_pad_in,
                                           B, k, V, W_in, &src, &dst, (int32_t*)d_tokens, (int32_t*)d_n_acc,
                                           (int32_t*)d_bonus, (int32_t*)d_pad_out, (int32_t*)d_w_new,
                                           (int64_t*)d_pos, (uint8_t*)d_mask, pm_cap, (const int32_t*)d_s_in,
                                           s_in_stride, (int32_t*)d_s_out, s_out_stride, pad_id, d_ws, ws_bytes,
                                           (uint32_t*)d_status, &w_host, NULL);
  if (st != SPECDEC_OK) { fprintf(stderr, "specdec_step: %s\n", specdec_last_error()); return 10 + (int)st; }
  if (hipDeviceSynchronize() != hipSuccess) return 7;

  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;
  fwrite(&w_host, 4, 1, out);
  write_back(out, d_tokens, (size_t)B * (k + 1) * 4);
  write_back(out, d_n_acc, n_b);
  write_back(out, d_bonus, n_b);
  write_back(out, d_pad_out, n_b);
  write_back(out, d_w_new, 4);
  write_back(out, d_status, 4);
  write_back(out, d_dst, n_kv);
  write_back(out, d_pos, (size_t)B * pm_cap * 8);
  write_back(out, d_mask, (size_t)B * pm_cap);
  write_back(out, d_s_out, n_s_out);
  fclose(out);
  printf("ok\n");
  return 0;
}
"""


@pytest.mark.parametrize("in_place", [False, True], ids=["oop", "inplace"])
def test_fused_step_from_c(tmp_path, in_place):
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    exe = tmp_path / "step"
    (tmp_path / "step.c").write_text(PROGRAM)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    f"-I{ROOT / 'include'}", str(tmp_path / "step.c"), f"-L{LIB_DIR}", "-lspecdec",
                    f"-Wl,-rpath,{LIB_DIR}", "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                    "-o", str(exe)], check=True)

    w = wl.WORKLOADS["vicuna7b"].scaled(L=2, H=4, prompt=("uniform", 100, 700))
    seed = 3
    n, W_in, pad_in, cap = wl.initial_geometry(w, seed)
    logits, draft, *_ = wl.logits_and_drafts(w, seed, 0, device="cpu")
    src = wl.make_kv(w, pad_in, W_in, cap, seed, device="cpu")
    s_in_stride, s_out_stride, pm_cap = cap + 2, (cap + 2 if in_place else W_in + 1 + 3), W_in + w.k + 1 + 5
    s_in = wl.make_token_rows(w, pad_in, W_in, s_in_stride, seed, PAD_ID, device="cpu")
    kv_bits = src.view(torch.int16).numpy().view(np.uint16)
    header = np.array([w.B, w.k, w.V, W_in, w.L, w.H, w.D, cap, pm_cap, s_in_stride, s_out_stride, PAD_ID,
                       int(in_place)], np.int32)
    with open(tmp_path / "in.bin", "wb") as f:
        for a in (header, logits.view(torch.int16).numpy(), draft.numpy().astype(np.int32),
                  np.asarray(pad_in, np.int32), kv_bits, s_in.numpy().astype(np.int32)):
            f.write(np.ascontiguousarray(a).tobytes())
    say(f"C program: B={w.B} k={w.k} V={w.V} L={w.L} H={w.H} D={w.D} W_in={W_in} cap={cap} in_place={in_place}")
    r = subprocess.run([str(exe), str(tmp_path / "in.bin"), str(tmp_path / "out.bin")], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr

    B, k = w.B, w.k
    buf = (tmp_path / "out.bin").read_bytes()
    off = 0

    def take(dtype, count):
        nonlocal off
        a = np.frombuffer(buf, dtype=dtype, count=count, offset=off)
        off += a.nbytes
        return a

    w_host = int(take(np.int32, 1)[0])
    tokens = take(np.int32, B * (k + 1)).reshape(B, k + 1)
    n_acc, bonus, pad_out = take(np.int32, B), take(np.int32, B), take(np.int32, B)
    w_new, status = int(take(np.int32, 1)[0]), int(take(np.uint32, 1)[0])
    dst = take(np.uint16, kv_bits.size).reshape(kv_bits.shape)
    pos = take(np.int64, B * pm_cap).reshape(B, pm_cap)
    mask = take(np.uint8, B * pm_cap).reshape(B, pm_cap)
    s_out = take(np.int32, B * s_out_stride).reshape(B, s_out_stride)
    assert off == len(buf)

    v = oracle.verify(logits, w.logit_dtype, draft.numpy(), pad_in, W_in)
    assert status == 0
    assert np.array_equal(tokens, v["tokens"]) and np.array_equal(n_acc, v["n_acc"])
    assert np.array_equal(bonus, v["bonus"]) and np.array_equal(pad_out, v["pad_out"])
    W = v["w_new"]
    assert w_new == W and w_host == W
    exp = oracle.realign_kv(kv_bits, k, W_in, pad_in, v["n_acc"], W)
    assert np.array_equal(dst[..., :W, :], exp[..., :W, :]), "cache differs from the oracle"
    if not in_place:
        assert np.all(dst[..., W:, :] == 0x7F7F), "cache columns beyond L' were written"
    epos, emask = oracle.posmask(v["pad_out"], W, k, pm_cap)
    width = W + k + 1
    assert np.array_equal(pos[:, :width], epos[:, :width]) and np.array_equal(mask[:, :width], emask[:, :width])
    assert np.all(pos[:, width:] == 0x6666666666666666) and np.all(mask[:, width:] == 0x77)
    es = oracle.realign_tokens(s_in.numpy(), v["tokens"], pad_in, v["n_acc"], W, W_in, PAD_ID)
    assert np.array_equal(s_out[:, :W + 1], es[:, :W + 1]), "token row differs from the oracle"
    if not in_place:
        assert np.all(s_out[:, W + 1:] == 0x55555555)
