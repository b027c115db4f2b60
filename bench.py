#!/usr/bin/env python3
"""Benchmark of one greedy verify + KV realign step (EqSpec) on one MI355X.

A step is one call of the fused ``specdec_step`` (the two verify kernels,
then the realign kernel with the position ids / mask and the token row S
fused in) over one batch of synthetic input already resident in HBM.  The default workload is the
Vicuna-7B-shaped batch (B=8, k=5, V=32000 bf16 logits; KV L=32, H=32, D=128
bf16; prompts U[128,1024]; out-of-place realign).

Prints ONE JSON line on stdout: steps/s, ms/step, the realign kernel's
achieved HBM bandwidth against the 8 TB/s peak (timed with HIP events the
library records on the launch stream), the HBM traffic measured by rocprofv3
counters when the committed summary matches the current kernel source, and
the CPU oracle timed on a bounded sample of the same step.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--variant oop|inplace]
                  [--noalloc] [--graph | --bound]
  python bench.py --path exspec [--exspec-batch ragged|same]
  python bench.py --verify sample [--temperature T]
  python bench.py --path varlen        # Family B rollback of a flat cache
  python bench.py --path chained       # 16 chained in-place steps (per-step times)
  python bench.py --path verify [--workload NAME]   # greedy verification alone, cold and warm caches
  python bench.py --copy-calibration GIB   # plain device copy, for counter scaling

``--path exspec`` measures EXSpec's step instead (Algorithm 2 without the
model forwards): the batch gather from a sequence pool (with the fused token
rows, paddings and position ids / mask), greedy verification, and the
append-only write-back, on the same shapes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

PEAK_HBM_GBS = 8000.0
WHOLE_STEP_MAX_BYTES = 16 << 30   # the CPU baseline runs one whole oracle step when the cache is at most this
METRIC = "verify+realign steps/s and achieved HBM GB/s (% peak), B=8 7B-shaped KV"
METRIC_EXSPEC = "EXSpec gather+verify+write-back steps/s and achieved HBM GB/s (% peak), B=8 7B-shaped KV"
METRIC_SAMPLE = "stochastic verify+realign steps/s and achieved HBM GB/s (% peak), B=8 7B-shaped KV"
METRIC_VARLEN = "variable-length rollback steps/s and achieved HBM GB/s (% peak), B=8 7B-shaped KV"
METRIC_VERIFY = "greedy verification calls/s from cold caches and achieved HBM GB/s (% peak) of the vocabulary scan"
METRIC_VERIFY_SAMPLE = ("stochastic verification calls/s from cold caches and achieved HBM GB/s (% peak) of the "
                        "row statistics")
CSRC = ROOT / "paper_2510_22876_amd" / "csrc"
KERNEL_SRCS = [CSRC / f for f in ("specdec_kernels.hip", "span_copy.h", "posmask.h")]
GATHER_SRCS = [CSRC / f for f in ("exspec_kernels.hip", "span_copy.h", "posmask.h")]
VARLEN_SRCS = [CSRC / f for f in ("rollback_kernels.hip", "span_copy.h")]
SAMPLE_SRCS = [CSRC / "sample_kernels.hip"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(srcs=None) -> str:
    """Hash of the sources the measured kernel is built from."""
    h = hashlib.sha256()
    for f in srcs or KERNEL_SRCS:
        h.update(f.read_bytes())
    return h.hexdigest()[:16]


def describe(w, variant):
    p = w.prompt
    pr = f"U[{p[1]},{p[2]}]" if p[0] == "uniform" else (f"log-U[{p[1]},{p[2]}]" if p[0] == "loguniform" else str(p))
    return (f"{w.name}: B={w.B} k={w.k} V={w.V} {w.logit_dtype} logits; KV L={w.L} H={w.H} D={w.D} bf16; "
            f"prompts {pr}; accept {w.accept[0]}; {'out-of-place' if variant == 'oop' else 'in-place'} realign")


def step_bytes(w, pad_in, W_in, n_acc, w_new, variant, token_row=True):
    """Algorithmic bytes of one step: what the method must read and write."""
    C = w.column_bytes
    W0 = W_in - (w.k + 1)
    lens = (W0 - pad_in.astype(np.int64)) + n_acc.astype(np.int64) + 1
    pad_out = w_new - lens
    shift = pad_out - pad_in
    if variant == "oop":
        realign = int(lens.sum()) * C + w.B * w_new * C
    else:
        moved = shift != 0
        realign = int(2 * lens[moved].sum()) * C + int(np.clip(shift, 0, None).sum()) * C
    posmask = w.B * (w_new + w.k + 1) * (8 + 1)
    if token_row:   # read each row's c_i + 1 tokens and n_acc + 1 predictions, write w_new + 1 columns
        posmask += 4 * int((lens - n_acc.astype(np.int64)).sum()) + 4 * int((n_acc.astype(np.int64) + 1).sum()) \
            + 4 * w.B * (w_new + 1)
    verify = w.B * (w.k + 1) * w.V * w.logit_bytes + 4 * w.B * w.k + 4 * w.B \
        + 4 * w.B * (w.k + 1) + 3 * 4 * w.B + 4
    return dict(realign=realign, posmask=posmask, verify=verify)


def read_traffic_summary(workload: str, variant: str, alg_bytes: int, kernel: str = "realign", srcs=None):
    """HBM bytes per launch of the measured kernel from the committed rocprofv3
    counter summary, if it was taken on the current kernel source and on a
    launch with the same algorithmic bytes as this run's (the same step)."""
    path = ROOT / "profiles" / f"{kernel}_{variant}_{workload}_hbm_counters.md"
    if not path.exists():
        return None, "no counter summary"
    text = path.read_text()
    m_hash = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    m_alg = re.search(r"Algorithmic bytes per launch \(bench.py\):\s*(\d+)", text)
    if not m_hash or not m_bytes or not m_alg:
        return None, "summary unreadable"
    if m_hash.group(1) != kernel_source_hash(srcs):
        return None, "kernel changed since the counters were taken"
    if int(m_alg.group(1)) != int(alg_bytes):
        return None, f"counters taken on another step ({m_alg.group(1)} algorithmic bytes)"
    return float(m_bytes.group(1)), path.name


def oracle_threads(layer_job, budget_s: float, L: int, serial_s: float):
    """The same oracle calls on N host threads at once (ctypes releases the
    GIL), one layer slab per call: N = min(16, cores), each thread calling
    until about ``budget_s / 2`` seconds have passed (at least once); the
    per-step time is the serial part (verification, pos/mask, token row) plus
    L layers at the measured per-layer rate."""
    from concurrent.futures import ThreadPoolExecutor
    n = max(1, min(16, os.cpu_count() or 1))
    if n == 1:
        return None
    t0 = time.perf_counter()
    deadline = t0 + budget_s / 2

    def worker(t):
        c = 0
        while True:
            layer_job(t + c * n)
            c += 1
            if time.perf_counter() >= deadline:
                return c

    with ThreadPoolExecutor(max_workers=n) as ex:
        calls = sum(ex.map(worker, range(n)))
    wall = time.perf_counter() - t0
    est = serial_s + wall / calls * L
    return dict(value=1.0 / est, unit="steps/s", cores=n, sample=f"{calls} one-layer calls on {n} threads")


def cpu_info() -> dict:
    """The host CPU as /proc/cpuinfo describes it: the full model name, the
    cache size line, family / model / stepping, and the logical CPUs seen."""
    info = {"model": "unknown", "cache": "unknown", "family_model_stepping": "unknown", "logical_cpus": 0}
    fms = {}
    try:
        for ln in Path("/proc/cpuinfo").read_text().splitlines():
            key, _, val = ln.partition(":")
            key, val = key.strip(), val.strip()
            if key == "processor":
                info["logical_cpus"] += 1
            elif key == "model name" and info["model"] == "unknown":
                info["model"] = val
            elif key == "cache size" and info["cache"] == "unknown":
                info["cache"] = val
            elif key in ("cpu family", "model", "stepping") and key not in fms:
                fms[key] = val
    except OSError:
        pass
    if fms:
        info["family_model_stepping"] = "/".join(fms.get(k, "?") for k in ("cpu family", "model", "stepping"))
    return info


def cpu_fields() -> dict:
    """The cpu_baseline fields that name the host CPU."""
    ci = cpu_info()
    return dict(cpu_model=ci["model"], cpu_cache=ci["cache"], cpu_family_model_stepping=ci["family_model_stepping"],
                host_logical_cpus=ci["logical_cpus"])


def copy_ceiling(nbytes: int, reps: int = 5) -> float:
    """GB/s (bytes read + written) of the runtime's device-to-device memcpy
    (``Tensor.copy_`` of contiguous bytes, which HIP serves with its blit
    kernel) of ``nbytes`` each way on this GPU: the data-movement rate a
    caller gets without a hand-written kernel."""
    import torch
    n = max(1 << 20, int(nbytes))
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b.copy_(a)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    del a, b
    torch.cuda.empty_cache()
    return 2 * n / (ms * 1e-3) / 1e9


def percentiles(ms):
    a = np.sort(np.asarray(ms, dtype=np.float64))
    return {"step_ms_p10": round(float(np.percentile(a, 10)), 5), "step_ms_p50": round(float(np.percentile(a, 50)), 5),
            "step_ms_p90": round(float(np.percentile(a, 90)), 5)}


def cpu_baseline(w, logits, draft, pad_in, W_in, src, budget_s: float, s_rows=None, sample=None):
    """The oracle as it stands, single-threaded on the host: verification
    over every logit row (greedy, or stochastic when ``sample`` =
    (draft_logits, u_accept, u_sample, temperature)), position ids / mask and
    the token row, and the KV realignment, timed two ways: over the whole
    cache in one call (one whole step; when the cache is at most
    WHOLE_STEP_MAX_BYTES) and on a bounded sample of whole layer slabs
    (cycling over up to two layers until ``budget_s`` seconds of work) scaled
    to every layer.  The value is the whole step when it ran, else the
    estimate; the same layer calls on N host threads give ``threads``."""
    import oracle
    k = w.k
    lg = logits.cpu()
    dr = draft.cpu().numpy()
    t0 = time.perf_counter()
    if sample is None:
        v = oracle.verify(lg, w.logit_dtype, dr, pad_in, W_in)
    else:
        dlg, ua, us, temp = sample
        v = oracle.verify_sample(lg, dlg.cpu(), w.logit_dtype, dr, pad_in, ua.cpu().numpy(), us.cpu().numpy(),
                                 temp, W_in)
    t_verify = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.posmask(v["pad_out"], v["w_new"], k)
    if s_rows is not None:
        oracle.realign_tokens(s_rows, v["tokens"], pad_in, v["n_acc"], v["w_new"], W_in, -1)
    t_pm = time.perf_counter() - t0
    nl = min(w.L, 2)
    slabs = [src[l:l + 1, :, :, :, :W_in, :].contiguous() for l in range(nl)]
    import torch
    host = [s.view(torch.int16).cpu().numpy().view(np.uint16) for s in slabs]
    runs = 0
    t_real = 0.0
    while t_real < budget_s or runs == 0:
        h = host[runs % nl]
        t0 = time.perf_counter()
        oracle.realign_kv(h, k, W_in, pad_in, v["n_acc"], v["w_new"])
        t_real += time.perf_counter() - t0
        runs += 1
    per_layer = t_real / runs
    est = t_verify + per_layer * w.L + t_pm
    mt = oracle_threads(lambda i: oracle.realign_kv(host[i % nl], k, W_in, pad_in, v["n_acc"], v["w_new"]),
                        budget_s, w.L, t_verify + t_pm)
    del host, slabs
    # one whole step, every layer in one oracle call, when the cache (and the
    # oracle's output of the same size) fits comfortably in host memory
    whole = None
    cache_bytes = w.L * 2 * w.B * w.H * W_in * w.D * 2
    if cache_bytes <= WHOLE_STEP_MAX_BYTES:
        full = src[:, :, :, :, :W_in, :].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        t0 = time.perf_counter()
        oracle.realign_kv(full, k, W_in, pad_in, v["n_acc"], v["w_new"])
        t_full = time.perf_counter() - t0
        del full
        whole = t_verify + t_full + t_pm
    value = 1.0 / whole if whole is not None else 1.0 / est
    return dict(value=value, unit="steps/s", cores=1, kind="oracle", **cpu_fields(),
                whole_step_s=round(whole, 4) if whole is not None else None, sampled_estimate_s=round(est, 4),
                threads=mt,
                sample=(f"oracle {'stochastic ' if sample is not None else ''}verify over all "
                        f"{w.B * (w.k + 1) + (w.B * w.k if sample is not None else 0)} logit rows ({t_verify * 1e3:.1f} ms), "
                        + (f"KV realign of the whole {cache_bytes / 1e9:.2f} GB cache in one call "
                           f"({(whole - t_verify - t_pm) * 1e3:.1f} ms), pos/mask and token row ({t_pm * 1e3:.2f} ms): "
                           f"one whole step single-threaded ({whole:.3f} s); the estimate from " if whole is not None
                           else "KV realign estimated from ")
                        + f"{runs} one-layer slabs cycling over layers 0..{nl - 1} ({per_layer * 1e3:.1f} ms per layer, "
                        f"x{w.L} layers) gives {est:.3f} s" + ("" if whole is not None else " (value)")))


def exspec_bytes(w, lens_b, Lb, n_acc):
    """Algorithmic bytes of EXSpec's step: the gather reads each row's cached
    entries and writes the padded batch (plus token rows and position ids /
    mask), the append write-back moves each row's n_acc + 1 new entries, and
    verification reads the logits."""
    C = w.column_bytes
    B, k = w.B, w.k
    lens_b = lens_b.astype(np.int64)
    a = n_acc.astype(np.int64) + 1
    gather = int(lens_b.sum()) * C + B * Lb * C
    gather_small = 4 * int((lens_b + 1).sum()) + 4 * B * (Lb + 1) + 9 * B * (Lb + k + 1) + 4 * 2 * B + 4 * B
    writeback = 2 * int(a.sum()) * C + 4 * int(a.sum()) * 2 + 4 * B * (k + 1) + 4 * 4 * B
    verify = B * (k + 1) * w.V * w.logit_bytes + 4 * B * k + 4 * B + 4 * B * (k + 1) + 3 * 4 * B + 4
    return dict(gather=gather + gather_small, writeback=writeback, verify=verify)


def cpu_baseline_exspec(w, pool, pool_tok, lens, slots, Lb, logits, draft, budget_s):
    """The oracle, single-threaded, on a bounded sample of EXSpec's step:
    verification over every logit row, and the gather and (whole-row)
    write-back of one-layer slabs of the pool cycling over up to two layers
    until ``budget_s`` seconds of work; scaled to one whole step."""
    import oracle
    import torch
    k = w.k
    bcap = Lb + k + 1
    host_pool = [pool[l:l + 1].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                 for l in range(min(w.L, 2))]
    tok = pool_tok.cpu().numpy()
    t0 = time.perf_counter()
    v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), np.asarray(Lb - lens[slots], np.int32),
                      Lb + k + 1)
    t_verify = time.perf_counter() - t0
    runs, t_layers = 0, 0.0
    while t_layers < budget_s or runs == 0:
        hp = host_pool[runs % len(host_pool)].copy()
        ln = lens.copy()
        tk = tok.copy()
        t0 = time.perf_counter()
        batch, btok, pads = oracle.gather_batch(hp, tk, ln, slots, Lb, bcap, bcap + 1, -1)
        oracle.scatter_accepted(batch, pads, v["tokens"], v["n_acc"], slots, Lb, hp, tk, ln)
        t_layers += time.perf_counter() - t0
        runs += 1
    per_layer = t_layers / runs
    est = t_verify + per_layer * w.L
    return dict(value=1.0 / est, unit="steps/s", cores=1, kind="oracle", **cpu_fields(),
                sample=(f"oracle verify over all {w.B * (k + 1)} logit rows ({t_verify * 1e3:.1f} ms), gather + "
                        f"whole-row write-back of {runs} one-layer pool slabs ({per_layer * 1e3:.1f} ms per layer, "
                        f"x{w.L} layers); single-threaded, scaled to one whole step ({est:.2f} s)"))


def bench_exspec(args, w):
    """EXSpec's step on one GPU: gather a batch of B rows from a pool of 4B
    sequences, verify it, write the accepted entries back (append mode)."""
    import torch
    from paper_2510_22876_amd import specdec as sd
    from paper_2510_22876_amd import workloads as wl

    B, k = w.B, w.k
    N = 4 * B
    lens = wl.pool_lengths(w, N, args.seed)
    if args.exspec_batch == "same":
        lens[:B] = lens[0]                      # a same-length group: the batch is a plain concatenation
    slots = np.arange(B, dtype=np.int32)        # the batch: the pool's first B sequences
    Lb = int(lens[:B].max())
    cap = int(lens.max()) + 2 * (k + 1)
    pool, pool_tok = wl.make_pool(w, lens, cap, cap + 2, args.seed, device="cuda")
    bcap = Lb + k + 1
    batch = torch.empty((w.L, 2, B, w.H, bcap, w.D), dtype=torch.bfloat16, device="cuda")
    btok = torch.empty((B, bcap + 1), dtype=torch.int32, device="cuda")
    pads = torch.empty(B, dtype=torch.int32, device="cuda")
    pos = torch.empty((B, bcap), dtype=torch.int64, device="cuda")
    mask = torch.empty((B, bcap), dtype=torch.uint8, device="cuda")
    logits, draft, *_ = wl.logits_and_drafts(w, args.seed, 0, device="cuda")
    bufs = sd.StepBuffers(B, k, w.V, bcap, "cuda")
    lens_d = torch.as_tensor(lens, device="cuda")
    lens0 = lens_d.clone()
    slots_d = torch.as_tensor(slots, device="cuda")
    status = bufs.dev_status
    W_in = Lb + k + 1
    desc = (f"{w.name} pool: N={N} sequences, lengths {w.prompt}; batch: slots 0..{B - 1} "
            f"({'same length' if args.exspec_batch == 'same' else 'ragged, unpad-repad'}), Lb={Lb}; B={B} k={k} "
            f"V={w.V} {w.logit_dtype} logits; KV L={w.L} H={w.H} D={w.D} bf16; append write-back")
    log(f"[bench] exspec: {desc}")

    def step():
        sd.specdec_gather_batch(pool, pool_tok, lens_d, slots_d, Lb, batch, pads, batch_tok=btok, pos=pos, mask=mask,
                                k=k, pad_id=-1, dev_status=status)
        sd.specdec_verify_greedy(logits, draft, pads, W_in, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out,
                                 bufs.w_new, bufs.workspace, status)
        sd.specdec_scatter_accepted(batch, pads, bufs.tokens, bufs.n_acc, slots_d, Lb, pool, pool_tok, lens_d,
                                    batch_tok=btok, mode=sd.WRITEBACK_APPEND, dev_status=status)

    def timed_pass(K, mask_bits):
        # the write-back grows each slot's length: restore it before every
        # step, outside the events that bracket the step
        sd.timing_reset()
        sd.timing_enable(mask_bits)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        total = 0.0
        for _ in range(K):
            lens_d.copy_(lens0)
            s.record()
            step()
            e.record()
            torch.cuda.synchronize()
            total += s.elapsed_time(e) / 1e3
        sd.timing_enable(False)
        return total

    timed_pass(args.warmup, 0)
    if int(status.cpu()[0]) != 0:
        raise RuntimeError("device flagged invalid values")
    n_acc = bufs.n_acc.cpu().numpy()
    K = args.steps
    elapsed = timed_pass(K, 1 << sd.KERNEL_GATHER)
    gather_ms, gather_n = sd.timing_query(sd.KERNEL_GATHER)
    timed_pass(K, (1 << sd.KERNEL_VERIFY) | (1 << sd.KERNEL_WRITEBACK))
    verify_ms, verify_n = sd.timing_query(sd.KERNEL_VERIFY)
    wb_ms, wb_n = sd.timing_query(sd.KERNEL_WRITEBACK)
    assert gather_n == K and verify_n == K and wb_n == K
    by = exspec_bytes(w, lens[:B], Lb, n_acc)
    g_ms = gather_ms / K
    achieved = by["gather"] / (g_ms * 1e-3) / 1e9
    ms_per_step = elapsed / K * 1e3
    total_bytes = by["gather"] + by["writeback"] + by["verify"]
    variant = "same" if args.exspec_batch == "same" else "ragged"
    traffic, traffic_src = read_traffic_summary(w.name, variant, by["gather"], kernel="gather", srcs=GATHER_SRCS)
    log(f"[bench] exspec n_acc={n_acc.tolist()} gather {g_ms:.4f} ms ({by['gather'] / 1e9:.3f} GB, {achieved:.0f} GB/s), "
        f"verify {verify_ms / K:.4f} ms, write-back {wb_ms / K:.4f} ms ({by['writeback'] / 1e6:.2f} MB), "
        f"step {ms_per_step:.4f} ms; traffic: {traffic_src}")
    cpu = None
    if args.cpu_baseline_seconds > 0:
        cpu = cpu_baseline_exspec(w, pool, pool_tok, lens, slots, Lb, logits, draft, args.cpu_baseline_seconds)
        log(f"[bench] cpu baseline: {cpu['value']:.4f} steps/s ({cpu['sample']})")
    line = {
        "metric": METRIC_EXSPEC,
        "value": K / elapsed,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": desc, "B": B, "k": k, "V": w.V, "L": w.L, "H": w.H, "D": w.D, "N": N, "Lb": Lb,
            "batch": variant, "seed": args.seed, "step_bytes": total_bytes,
            "step_GBps": round(total_bytes / (ms_per_step * 1e-3) / 1e9, 1),
            "gather_ms": round(g_ms, 5), "verify_ms": round(verify_ms / K, 5), "writeback_ms": round(wb_ms / K, 5),
        },
        "roofline": {
            "bound": "hbm", "kernel": "gather (+ fused token rows, pos/mask)", "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
            "algorithmic_bytes": by["gather"],
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def bench_varlen(args, w):
    """Family B rollback on one GPU: the workload's sequences (cached entries
    from its prompt distribution, plus the k+1 window rows each) in a flat
    [L][2][T][H][D] cache, greedy verification, then the compaction that rolls
    back each sequence's rejected window rows into a second buffer, with the
    new offsets and position ids."""
    import torch
    from paper_2510_22876_amd import specdec as sd
    from paper_2510_22876_amd import workloads as wl

    B, k = w.B, w.k
    n = wl.prompt_lengths(w, args.seed)
    lens = n + k + 1
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed + 12345)
    src = torch.randn((w.L, 2, T, w.H, w.D), generator=g, device="cuda").to(torch.bfloat16)
    dst = torch.empty_like(src)
    logits, draft, *_ = wl.logits_and_drafts(w, args.seed, 0, device="cuda")
    bufs = sd.StepBuffers(B, k, w.V, 8, "cuda")
    cu_d = torch.as_tensor(cu, device="cuda")
    cu_out = torch.empty(B + 1, dtype=torch.int32, device="cuda")
    pos = torch.empty(T, dtype=torch.int64, device="cuda")
    zeros = torch.zeros(B, dtype=torch.int32, device="cuda")
    max_len = int(lens.max())
    desc = (f"{w.name} as a flat cache: B={B} sequences, cached lengths {w.prompt} + k+1={k + 1} window rows, "
            f"T={T}; k={k} V={w.V} {w.logit_dtype} logits; KV L={w.L} H={w.H} D={w.D} bf16; out-of-place compaction")
    log(f"[bench] varlen: {desc}")

    def step():
        sd.specdec_verify_greedy(logits, draft, zeros, k + 1, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out,
                                 bufs.w_new, bufs.workspace, bufs.dev_status)
        sd.specdec_varlen_rollback(src, dst, cu_d, bufs.n_acc, k, max_len, cu_out, pos, bufs.dev_status)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if int(bufs.dev_status.cpu()[0]) != 0:
        raise RuntimeError("device flagged invalid values")
    n_acc = bufs.n_acc.cpu().numpy()
    K = args.steps
    sd.timing_reset()
    sd.timing_enable(1 << sd.KERNEL_VARLEN)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    sd.timing_enable(False)
    v_ms, v_n = sd.timing_query(sd.KERNEL_VARLEN)
    assert v_n == K
    E = w.L * 2 * w.H * w.D * 2
    keep = lens - (k - n_acc)
    algo = 2 * int(keep.sum()) * E + 4 * (2 * B + 1) + 4 * B + 8 * int(keep.sum())
    vms = v_ms / K
    achieved = algo / (vms * 1e-3) / 1e9
    ms_per_step = elapsed / K * 1e3
    traffic, traffic_src = read_traffic_summary(w.name, "oop", algo, kernel="varlen", srcs=VARLEN_SRCS)
    log(f"[bench] varlen n_acc={n_acc.tolist()} compaction {vms:.4f} ms ({algo / 1e9:.3f} GB, {achieved:.0f} GB/s), "
        f"step {ms_per_step:.4f} ms; traffic: {traffic_src}")
    cpu = None
    if args.cpu_baseline_seconds > 0:
        cpu = cpu_baseline_varlen(w, logits, draft, src, cu, args.cpu_baseline_seconds)
        log(f"[bench] cpu baseline: {cpu['value']:.4f} steps/s ({cpu['sample']})")
    line = {
        "metric": METRIC_VARLEN, "value": K / elapsed, "unit": "steps/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": desc, "B": B, "k": k, "V": w.V, "L": w.L, "H": w.H, "D": w.D, "T": T,
                   "seed": args.seed, "compaction_ms": round(vms, 5)},
        "roofline": {"bound": "hbm", "kernel": "varlen offsets + compaction (+ positions)", "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": algo},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def cpu_baseline_verify(w, logits, draft, pad_in, W_in, budget_s, sample=None):
    """The oracle's verification (every logit row; stochastic when ``sample``
    holds the draft logits, uniforms and temperature) on one host thread,
    called until ``budget_s`` seconds have passed (at least once)."""
    import oracle
    lg = logits.cpu()
    dr = draft.cpu().numpy()
    if sample:
        dl, ua, us, T = sample
        dl, ua, us = dl.cpu(), ua.cpu().numpy(), us.cpu().numpy()
    t0 = time.perf_counter()
    calls = 0
    while True:
        if sample:
            oracle.verify_sample(lg, dl, w.logit_dtype, dr, pad_in, ua, us, T, W_in)
        else:
            oracle.verify(lg, w.logit_dtype, dr, pad_in, W_in)
        calls += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    wall = time.perf_counter() - t0
    rows = w.B * ((2 * w.k + 1) if sample else (w.k + 1))
    return dict(value=calls / wall, unit="calls/s", cores=1, kind="oracle", **cpu_fields(),
                sample=f"{calls} whole oracle {'stochastic ' if sample else ''}verifications ({rows} logit rows each) "
                       f"in {wall:.2f} s")


def bench_verify(args, w):
    """Greedy verification alone (Algorithm 3 and Eq. (1)-(2): the two
    launches of specdec_verify_greedy) on the workload's logits.  Cold: before
    every timed call a 1 GiB buffer is read (a reduction outside the events),
    which evicts the 256 MB Infinity Cache and the L2s without leaving dirty
    lines behind, so the scan reads its logits from HBM.  Warm: before every
    call the GPU only waits (a bounded sleep kernel), so logits that fit the
    Infinity Cache stay there.  Either way the call is queued behind a
    kernel of some hundred microseconds, so the events time the GPU's work
    and not the host's submission.  The roofline is the scan kernel's (events
    around its launch alone); the line's value is cold calls per second of
    event time."""
    import torch
    from paper_2510_22876_amd import specdec as sd
    from paper_2510_22876_amd import workloads as wl

    n, W_in, pad_in, cap = wl.initial_geometry(w, args.seed)
    sample = args.verify == "sample"
    if sample:
        logits, draft_logits, draft, u_accept, u_sample = wl.sampled_inputs(w, args.seed, 0, device="cuda",
                                                                            temperature=args.temperature)
        sws = sd.alloc_sample_workspace(w.B, w.k, w.V)
        rows = w.B * (2 * w.k + 1)
    else:
        logits, draft, *_ = wl.logits_and_drafts(w, args.seed, 0, device="cuda")
        rows = w.B * (w.k + 1)
    bufs = sd.StepBuffers(w.B, w.k, w.V, 8, "cuda")
    pad_t = torch.as_tensor(pad_in, device="cuda")
    evict = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    kind = f"stochastic verification (T={args.temperature}, target and draft logits)" if sample else "verification"
    desc = (f"{w.name} {kind}: B={w.B} k={w.k} V={w.V} {w.logit_dtype} logits "
            f"({rows * w.V * w.logit_bytes / 1e6:.2f} MB), W_in={W_in}")
    log(f"[bench] verify: {desc}")

    def call():
        if sample:
            sd.specdec_verify_sample(logits, draft_logits, draft, pad_t, u_accept, u_sample, args.temperature, W_in,
                                     bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out, bufs.w_new, sws,
                                     bufs.dev_status)
        else:
            sd.specdec_verify_greedy(logits, draft, pad_t, W_in, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out,
                                     bufs.w_new, bufs.workspace, bufs.dev_status)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    if int(bufs.dev_status.cpu()[0]) != 0:
        raise RuntimeError("device flagged invalid values")
    K = args.steps
    whole, scan = (sd.KERNEL_SAMPLE, sd.KERNEL_SAMPLE_STATS) if sample else (sd.KERNEL_VERIFY, sd.KERNEL_VERIFY_SCAN)

    evict.fill_(1)
    sink = torch.empty(K, dtype=torch.int64, device="cuda")

    def timed_calls(cold: bool, kernel: int):
        # one timer per pass: a timer nested inside another would add its
        # events to the outer interval
        sd.timing_reset()
        sd.timing_enable(1 << kernel)
        for i in range(K):
            if cold:
                torch.sum(evict, dim=0, dtype=torch.int64, out=sink[i])
            else:
                torch.cuda._sleep(1 << 20)
            call()
        torch.cuda.synchronize()
        sd.timing_enable(False)
        ms, n = sd.timing_query(kernel)
        assert n == K
        return ms / K

    warm_ms, warm_scan_ms = timed_calls(False, whole), timed_calls(False, scan)
    cold_ms, cold_scan_ms = timed_calls(True, whole), timed_calls(True, scan)
    by = step_bytes(w, pad_in, W_in, bufs.n_acc.cpu().numpy(), int(bufs.w_new.cpu()[0]), "oop", False)
    scan_bytes = rows * w.V * w.logit_bytes
    achieved = scan_bytes / (cold_scan_ms * 1e-3) / 1e9
    traffic, traffic_src = read_traffic_summary(w.name, "cold", scan_bytes,
                                                kernel="samplestats" if sample else "verifyscan",
                                                srcs=SAMPLE_SRCS if sample else KERNEL_SRCS)
    log(f"[bench] verify cold {cold_ms * 1e3:.2f} us (scan {cold_scan_ms * 1e3:.2f} us, {achieved:.0f} GB/s), "
        f"warm {warm_ms * 1e3:.2f} us (scan {warm_scan_ms * 1e3:.2f} us); traffic: {traffic_src}")
    cpu = None
    if args.cpu_baseline_seconds > 0:
        cpu = cpu_baseline_verify(w, logits, draft, pad_in, W_in, args.cpu_baseline_seconds,
                                  sample=(draft_logits, u_accept, u_sample, args.temperature) if sample else None)
        log(f"[bench] cpu baseline: {cpu['value']:.2f} calls/s ({cpu['sample']})")
    line = {
        "metric": METRIC_VERIFY_SAMPLE if sample else METRIC_VERIFY, "value": 1e3 / cold_ms, "unit": "calls/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": cold_ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.logit_dtype, "data": "synthetic",
        "config": {"workload": desc, "B": w.B, "k": w.k, "V": w.V, "seed": args.seed,
                   "verify_cold_ms": round(cold_ms, 5), "verify_warm_ms": round(warm_ms, 5),
                   "scan_cold_ms": round(cold_scan_ms, 5), "scan_warm_ms": round(warm_scan_ms, 5),
                   "scan_warm_GBps": round(scan_bytes / (warm_scan_ms * 1e-3) / 1e9, 1),
                   "verify_bytes": by["verify"], "eviction_bytes": evict.numel()},
        "roofline": {"bound": "hbm", "kernel": ("sample_stats (row statistics of target and draft logits)" if sample
                                                else "verify_partial (vocabulary scan)") + ", cold caches",
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic, "algorithmic_bytes": scan_bytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def cpu_baseline_varlen(w, logits, draft, src, cu, budget_s):
    """The oracle, single-threaded, on a bounded sample of the Family B step:
    verification over every logit row, then the compaction of one-layer slabs
    of the flat cache cycling over up to two layers until ``budget_s`` seconds
    of work; scaled to one whole step."""
    import oracle
    import torch
    k = w.k
    t0 = time.perf_counter()
    v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), np.zeros(w.B, np.int32), k + 1)
    t_verify = time.perf_counter() - t0
    host = [src[l:l + 1].contiguous().view(torch.int16).cpu().numpy().view(np.uint16) for l in range(min(w.L, 2))]
    runs, t_layers = 0, 0.0
    while t_layers < budget_s or runs == 0:
        t0 = time.perf_counter()
        oracle.varlen_rollback(host[runs % len(host)], cu, v["n_acc"], k)
        t_layers += time.perf_counter() - t0
        runs += 1
    per_layer = t_layers / runs
    est = t_verify + per_layer * w.L
    return dict(value=1.0 / est, unit="steps/s", cores=1, kind="oracle", **cpu_fields(),
                sample=(f"oracle verify over all {w.B * (k + 1)} logit rows ({t_verify * 1e3:.1f} ms), compaction of "
                        f"{runs} one-layer slabs of the flat cache ({per_layer * 1e3:.1f} ms per layer, x{w.L} layers); "
                        f"single-threaded, scaled to one whole step ({est:.2f} s)"))


def bench_chained(args, w):
    """Chained in-place steps (the cache grows by the accepted entries each
    step): every step verifies fresh logits, realigns the cache and token row
    in place and writes the next verify window's entries (outside the timed
    intervals). K timed steps run through the chain of ``w.steps`` steps,
    restarting from the pristine input after the last; per-chain-step times
    and bandwidths are reported."""
    import torch
    from paper_2510_22876_amd import specdec as sd
    from paper_2510_22876_amd import workloads as wl
    k, B, T = w.k, w.B, w.steps
    n, W_in0, pad_in0, cap = wl.initial_geometry(w, args.seed)
    desc = describe(w, "inplace") + f"; {T} chained steps, cap={cap}"
    log(f"[bench] chained workload {desc}")
    kv = wl.make_kv(w, pad_in0, W_in0, cap, args.seed, device="cuda")
    pristine = kv.clone()
    s_rows = wl.make_token_rows(w, pad_in0, W_in0, cap + 2, args.seed, -1, device="cuda")
    pristine_s = s_rows.clone()
    inputs = [wl.logits_and_drafts(w, args.seed, t, device="cuda")[:2] for t in range(T)]
    bufs = sd.StepBuffers(B, k, w.V, cap + k + 1)
    st = dict(t=0, W0=W_in0 - (k + 1), pad=pad_in0.copy())
    pad_t = torch.as_tensor(pad_in0, device="cuda")

    def restart():
        kv.copy_(pristine)
        s_rows.copy_(pristine_s)
        pad_t.copy_(torch.as_tensor(pad_in0, device="cuda"))
        st.update(t=0, W0=W_in0 - (k + 1), pad=pad_in0.copy())

    def one(record=None):
        """One chained step; returns (chain position, bytes dict, realign ms)."""
        t = st["t"]
        if t == T:
            restart()
            t = 0
        if t > 0:
            wl.write_window(kv, w, st["W0"], st["pad"], seed=args.seed, step=t)
        Wi = st["W0"] + k + 1
        logits, draft = inputs[t]
        torch.cuda.synchronize()
        if record:
            record[0].record()
        sd.specdec_step(logits, draft, pad_t, Wi, kv, kv, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out,
                        bufs.w_new, bufs.pos, bufs.mask, bufs.workspace, bufs.dev_status, s_in=s_rows,
                        s_out=s_rows, pad_id=-1)
        if record:
            record[1].record()
        torch.cuda.synchronize()
        n_acc = bufs.n_acc.cpu().numpy()
        w_new = int(bufs.w_new.cpu()[0])
        by = step_bytes(w, st["pad"], Wi, n_acc, w_new, "inplace", True)
        st.update(t=t + 1, W0=w_new, pad=bufs.pad_out.cpu().numpy().copy())
        pad_t.copy_(bufs.pad_out)
        return t, by

    for _ in range(args.warmup):
        one()
    if int(bufs.dev_status.cpu()[0]) != 0:
        raise RuntimeError("device flagged invalid values")
    restart()
    K = args.steps
    per = {t: [] for t in range(T)}
    realign = {t: [] for t in range(T)}
    bytes_at = {}
    elapsed = 0.0
    for _ in range(K):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        sd.timing_reset()
        sd.timing_enable(1 << sd.KERNEL_REALIGN)
        t, by = one(ev)
        sd.timing_enable(False)
        ms = ev[0].elapsed_time(ev[1])
        rms, rn = sd.timing_query(sd.KERNEL_REALIGN)
        assert rn == 1
        per[t].append(ms)
        realign[t].append(rms)
        bytes_at[t] = by
        elapsed += ms / 1e3
    done = [t for t in range(T) if per[t]]
    rbytes = sum((bytes_at[t]["realign"] + bytes_at[t]["posmask"]) * len(per[t]) for t in done)
    rms_total = sum(sum(realign[t]) for t in done)
    achieved = rbytes / (rms_total * 1e-3) / 1e9
    per_step = [{"step": t, "ms": round(float(np.mean(per[t])), 5), "realign_ms": round(float(np.mean(realign[t])), 5),
                 "realign_GBps": round((bytes_at[t]["realign"] + bytes_at[t]["posmask"]) /
                                       (np.mean(realign[t]) * 1e-3) / 1e9, 1)} for t in done]
    ms_all = [m for t in done for m in per[t]]
    log(f"[bench] chained: {K} steps, mean {elapsed / K * 1e3:.4f} ms, realign {achieved:.0f} GB/s")
    cpu = None
    if args.cpu_baseline_seconds > 0:
        # the oracle on the chain's first step (its geometry, logits and cache)
        cpu = cpu_baseline(w, inputs[0][0], inputs[0][1], pad_in0, W_in0, pristine, args.cpu_baseline_seconds,
                           pristine_s.cpu().numpy())
        cpu["sample"] = "the chain's first step: " + cpu["sample"]
        log(f"[bench] cpu baseline: {cpu['value']:.4f} steps/s ({cpu['sample']})")
    copy_gbs = copy_ceiling(rbytes // (2 * K)) if args.copy_ceiling else None
    line = {
        "metric": METRIC, "value": K / elapsed, "unit": "steps/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": elapsed / K * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": desc, "B": B, "k": k, "V": w.V, "L": w.L, "H": w.H, "D": w.D, "chain": T,
                   "variant": "inplace", "seed": args.seed, "token_row": True, **percentiles(ms_all),
                   "per_step": per_step},
        "roofline": {"bound": "hbm", "kernel": "realign_inplace (+ fused pos/mask, token row)",
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                     "algorithmic_bytes": int(rbytes // K),
                     **({"memcpy_d2d_GBps": round(copy_gbs, 1), "vs_memcpy_d2d": round(achieved / copy_gbs, 4)}
                        if copy_gbs else {})},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def copy_calibration(gib: float):
    import torch
    n = int(gib * (1 << 30))
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    reps = 10
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / reps
    print(json.dumps({"copy_bytes_each_way": n, "ms_per_copy": ms, "GBps_read_plus_write": 2 * n / ms / 1e6}))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vicuna7b")
    ap.add_argument("--variant", default="oop", choices=["oop", "inplace"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-token-row", action="store_true", help="leave the token row S out of the step")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=10.0,
                    help="seconds of oracle realign work for the CPU baseline (0: skip)")
    ap.add_argument("--kernel-timers", choices=["on", "off"], default="on",
                    help="record the library's HIP events around the realign kernel inside the timed region "
                         "(off: a second pass measures it)")
    ap.add_argument("--verify", choices=["greedy", "sample"], default="greedy",
                    help="greedy verification (default) or stochastic verification by speculative sampling")
    ap.add_argument("--temperature", type=float, default=1.0, help="--verify sample: the sampling temperature")
    ap.add_argument("--path", choices=["eqspec", "exspec", "varlen", "chained", "verify"], default="eqspec",
                    help="eqspec: the verify + realign step (default); exspec: gather + verify + write-back; "
                         "varlen: Family B rollback; chained: in-place steps along a chain (per-step times)")
    ap.add_argument("--exspec-batch", choices=["ragged", "same"], default="ragged",
                    help="exspec: a batch of prompt-distributed lengths (unpad-repad) or one length (concatenation)")
    ap.add_argument("--noalloc", action="store_true",
                    help="greedy steps through specdec_step_noalloc (library scratch; one-launch verification "
                         "for small batches)")
    ap.add_argument("--graph", action="store_true",
                    help="capture the step in a HIP graph once and replay it in the timed loop")
    ap.add_argument("--bound", action="store_true",
                    help="greedy eager steps through specdec.bind_step: the arguments checked and marshalled "
                         "once, each step one library call with the stored arguments")
    ap.add_argument("--copy-ceiling", type=int, choices=[0, 1], default=1,
                    help="also time the runtime's device-to-device memcpy of the realign's bytes, for comparison")
    ap.add_argument("--copy-calibration", type=float, default=0.0,
                    help="run a plain device copy of this many GiB each way and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: this step runs on a single MI355X and has no multi-GPU "
              f"path (asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)
        return

    from paper_2510_22876_amd import specdec as sd
    from paper_2510_22876_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    if args.path == "exspec":
        bench_exspec(args, w)
        return
    if args.path == "varlen":
        bench_varlen(args, w)
        return
    if args.path == "verify":
        bench_verify(args, w)
        return
    if args.path == "chained":
        bench_chained(args, w if w.steps > 1 else wl.WORKLOADS["vicuna7b_chained"])
        return
    variant = args.variant
    n, W_in, pad_in, cap = wl.initial_geometry(w, args.seed)
    log(f"[bench] workload {describe(w, variant)}; W_in={W_in} cap={cap}")
    sample = args.verify == "sample"
    if sample:
        logits, draft_logits, draft, u_accept, u_sample = wl.sampled_inputs(w, args.seed, 0, device="cuda",
                                                                            temperature=args.temperature)
    else:
        logits, draft, *_ = wl.logits_and_drafts(w, args.seed, 0, device="cuda")
    src = wl.make_kv(w, pad_in, W_in, cap, args.seed, device="cuda")
    pristine = None
    if variant == "oop":
        dst = torch.empty_like(src)
    else:
        dst = src
        pristine = src.clone()
    pm_cap = W_in + w.k + 1
    bufs = sd.StepBuffers(w.B, w.k, w.V, pm_cap)
    pad_t = torch.as_tensor(pad_in, device="cuda")
    token_row = not args.no_token_row
    s_in = s_out = None
    if token_row:
        s_in = wl.make_token_rows(w, pad_in, W_in, W_in + 1, args.seed, -1, device="cuda")
        s_out = torch.empty_like(s_in) if variant == "oop" else s_in
    pristine_s = s_in.clone() if (token_row and variant != "oop") else None

    sws = sd.alloc_sample_workspace(w.B, w.k, w.V) if sample else None
    bound = None
    if args.bound:
        if sample or args.graph:
            raise SystemExit("--bound applies to eager greedy steps")
        bound = sd.bind_step(logits, draft, pad_t, W_in, src, dst, bufs.tokens, bufs.n_acc, bufs.bonus,
                             bufs.pad_out, bufs.w_new, bufs.pos, bufs.mask, None if args.noalloc else bufs.workspace,
                             bufs.dev_status, s_in=s_in, s_out=s_out, pad_id=-1, noalloc=args.noalloc)

    def step():
        if bound is not None:
            bound()
        elif sample:
            sd.specdec_step_sample(logits, draft_logits, draft, pad_t, u_accept, u_sample, args.temperature, W_in,
                                   src, dst, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out, bufs.w_new, bufs.pos,
                                   bufs.mask, sws, bufs.dev_status, s_in=s_in, s_out=s_out, pad_id=-1)
        elif args.noalloc:
            sd.specdec_step_noalloc(logits, draft, pad_t, W_in, src, dst, bufs.tokens, bufs.n_acc, bufs.bonus,
                                    bufs.pad_out, bufs.w_new, bufs.pos, bufs.mask, bufs.dev_status, s_in=s_in,
                                    s_out=s_out, pad_id=-1)
        else:
            sd.specdec_step(logits, draft, pad_t, W_in, src, dst, bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out,
                            bufs.w_new, bufs.pos, bufs.mask, bufs.workspace, bufs.dev_status, s_in=s_in, s_out=s_out,
                            pad_id=-1)

    def restore():
        src.copy_(pristine)
        if pristine_s is not None:
            s_in.copy_(pristine_s)

    for _ in range(args.warmup):
        if pristine is not None:
            restore()
        step()
    torch.cuda.synchronize()
    n_acc = bufs.n_acc.cpu().numpy()
    w_new = int(bufs.w_new.cpu()[0])
    if int(bufs.dev_status.cpu()[0]) != 0:
        raise RuntimeError("device flagged invalid values")

    K = args.steps
    timers = args.kernel_timers == "on" and not args.graph
    run = step
    if args.graph:
        # the step captured once in a HIP graph and replayed: no host work per
        # step (kernel timers stay off inside the capture; the second pass
        # below times the kernels eagerly)
        sd.timing_enable(False)
        if pristine is not None:
            restore()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run = graph.replay
    sd.timing_reset()
    # only the dominant kernel is bracketed inside the timed region
    sd.timing_enable(1 << sd.KERNEL_REALIGN if timers else 0)
    step_ms = []
    if pristine is None:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(K):
            run()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    else:
        # in place is not idempotent: restore the input before each step,
        # outside the timed intervals (events bracket each step)
        elapsed = 0.0
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(K):
            restore()
            s.record()
            run()
            e.record()
            torch.cuda.synchronize()
            step_ms.append(s.elapsed_time(e))
            elapsed += step_ms[-1] / 1e3
    sd.timing_enable(False)
    realign_ms, realign_n = sd.timing_query(sd.KERNEL_REALIGN)
    # a second pass of K steps after the timed region: the verify kernels'
    # durations (and the realign kernel's when it was not timed above)
    sd.timing_reset()
    vkern = sd.KERNEL_SAMPLE if sample else sd.KERNEL_VERIFY
    sd.timing_enable((1 << vkern) | (0 if timers else 1 << sd.KERNEL_REALIGN))
    for _ in range(K):
        if pristine is not None:
            restore()
        step()
    torch.cuda.synchronize()
    sd.timing_enable(False)
    verify_ms, verify_n = sd.timing_query(vkern)
    if not timers:
        realign_ms, realign_n = sd.timing_query(sd.KERNEL_REALIGN)
    # the first verification kernel alone in a pass of its own (a timer nested
    # in the verification's would add its events to that interval)
    scan_kern = sd.KERNEL_SAMPLE_STATS if sample else sd.KERNEL_VERIFY_SCAN
    sd.timing_reset()
    sd.timing_enable(1 << scan_kern)
    for _ in range(K):
        if pristine is not None:
            restore()
        step()
    torch.cuda.synchronize()
    sd.timing_enable(False)
    scan_ms, scan_n = sd.timing_query(scan_kern)
    if pristine is None:
        # the per-step distribution: events around each step of a third,
        # back-to-back pass
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
        for s_ev, e_ev in evs:
            s_ev.record()
            run()
            e_ev.record()
        torch.cuda.synchronize()
        step_ms = [s_ev.elapsed_time(e_ev) for s_ev, e_ev in evs]
    assert realign_n == K and verify_n == K

    by = step_bytes(w, pad_in, W_in, n_acc, w_new, variant, token_row)
    if sample:
        # every target and draft logit is read once; inputs and outputs are a few KB
        by["verify"] = w.B * (2 * w.k + 1) * w.V * w.logit_bytes + 4 * w.B * (2 * w.k + 1) + 4 * w.B * (w.k + 5) + 4
    realign_avg_ms = realign_ms / realign_n
    verify_avg_ms = verify_ms / verify_n
    realign_bytes = by["realign"] + by["posmask"]
    achieved = realign_bytes / (realign_avg_ms * 1e-3) / 1e9
    ms_per_step = elapsed / K * 1e3
    step_gbs = (realign_bytes + by["verify"]) / (ms_per_step * 1e-3) / 1e9
    traffic, traffic_src = read_traffic_summary(w.name, variant + ("sample" if sample else ""), realign_bytes)
    copy_gbs = copy_ceiling(realign_bytes // 2) if args.copy_ceiling else None
    log(f"[bench] n_acc={n_acc.tolist()} w_new={w_new} realign {realign_avg_ms:.4f} ms "
        f"({realign_bytes / 1e9:.3f} GB, {achieved:.0f} GB/s), verify {verify_avg_ms:.4f} ms "
        f"({by['verify'] / 1e6:.2f} MB), step {ms_per_step:.4f} ms ({step_gbs:.0f} GB/s); traffic: {traffic_src}")

    cpu = None
    if args.cpu_baseline_seconds > 0:
        s_host = None
        if token_row:
            s_host = (pristine_s if pristine_s is not None else s_in).cpu().numpy()
        cpu = cpu_baseline(w, logits, draft, pad_in, W_in, pristine if pristine is not None else src,
                           args.cpu_baseline_seconds, s_host,
                           sample=(draft_logits, u_accept, u_sample, args.temperature) if sample else None)
        log(f"[bench] cpu baseline: {cpu['value']:.4f} steps/s ({cpu['sample']})")

    line = {
        "metric": METRIC_SAMPLE if sample else METRIC,
        "value": K / elapsed,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": describe(w, variant) + (f"; stochastic verification at T={args.temperature}, draft logits = "
                                                 f"target + N(0,1), drafts drawn from q" if sample else ""),
            "B": w.B, "k": w.k, "V": w.V, "L": w.L, "H": w.H, "D": w.D, "W_in": W_in, "w_new": w_new,
            "variant": variant, "seed": args.seed, "token_row": token_row, "verify": args.verify,
            "graph": bool(args.graph), "noalloc": bool(args.noalloc), "bound": bool(args.bound),
            **({"temperature": args.temperature, "draft_noise": 1.0} if sample else {}),
            "step_GBps": round(step_gbs, 1),
            "step_bytes": realign_bytes + by["verify"],
            "verify_ms": round(verify_avg_ms, 5),
            **({"verify_scan_ms": round(scan_ms / scan_n, 5)} if scan_n else {}),
            "realign_ms": round(realign_avg_ms, 5),
            **percentiles(step_ms),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "realign_" + variant + " (+ fused pos/mask" + (", token row)" if token_row else ")"),
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
            "algorithmic_bytes": realign_bytes,
            **({"memcpy_d2d_GBps": round(copy_gbs, 1), "vs_memcpy_d2d": round(achieved / copy_gbs, 4)} if copy_gbs else {}),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
