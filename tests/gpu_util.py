"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare it with the oracle on the same input bytes."""
from __future__ import annotations

import sys
from dataclasses import dataclass, field

import numpy as np
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests import checker

SENT_KV = 0x7FC1        # a bf16 NaN pattern: marks destination columns the step must not touch
SENT_POS = -7
SENT_MASK = 0xAB
SENT_TOK = -555
PAD_ID = -2


def say(*a):
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 bit patterns on the host."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def i16(t: torch.Tensor) -> torch.Tensor:
    return t.view(torch.int16)


@dataclass
class StepResult:
    w: wl.Workload
    W_in: int
    cap: int
    pad_in: np.ndarray
    logits: torch.Tensor
    draft: torch.Tensor
    src: torch.Tensor             # pre-step input (a clone when the step ran in place)
    dst: torch.Tensor
    out: dict                     # device outputs copied to host
    pm_cap: int
    variant: str = "oop"
    extra: dict = field(default_factory=dict)


def alloc_outputs(B, k, V, pm_cap, device="cuda"):
    from paper_2510_22876_amd import specdec as sd
    bufs = sd.StepBuffers(B, k, V, pm_cap, device)
    for t in (bufs.tokens, bufs.n_acc, bufs.bonus, bufs.pad_out, bufs.w_new):
        t.fill_(-99)
    bufs.pos.fill_(SENT_POS)
    bufs.mask.fill_(SENT_MASK)
    return bufs


def run_gpu(w: wl.Workload, seed: int = 0, variant: str = "oop", api: str = "step",
            tagged: bool = False, keep_src: bool = True, dst_cap: int | None = None,
            logits=None, draft=None, pad_in=None, W_in=None, src=None, tokens: str | None = None,
            s_rows=None) -> StepResult:
    """One step of the HIP path.  ``api`` = "step" (fused) or "split"
    (verify, realign and posmask entry points in turn).  ``tokens`` = "oop" or
    "inplace" also realigns the token row S (given as ``s_rows`` or drawn)."""
    from paper_2510_22876_amd import specdec as sd
    say(f"workload={w.name} B={w.B} k={w.k} V={w.V} L={w.L} H={w.H} D={w.D} seed={seed} "
        f"variant={variant} api={api} tagged={tagged}")
    if W_in is None:
        n, W_in, pad_in0, cap = wl.initial_geometry(w, seed)
        pad_in = pad_in0 if pad_in is None else pad_in
    else:
        cap = W_in + w.extra_cap
    if logits is None:
        logits, draft, *_ = wl.logits_and_drafts(w, seed, 0, device="cuda")
    if src is None:
        src = wl.make_kv(w, pad_in, W_in, cap, seed, device="cuda", tagged=tagged)
    if variant == "oop":
        dcap = dst_cap if dst_cap is not None else cap
        dst = torch.full((w.L, 2, w.B, w.H, dcap, w.D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        before = src
    else:
        dst = src
        before = src.clone() if keep_src else None
    pm_cap = W_in + w.k + 1 + 3
    o = alloc_outputs(w.B, w.k, w.V, pm_cap)
    pad_t = torch.as_tensor(np.asarray(pad_in, np.int32), device="cuda")
    s_in = s_out = s_before = None
    if tokens is not None:
        stride = cap + 2
        if s_rows is None:
            s_rows = wl.make_token_rows(w, pad_in, W_in, stride, seed, PAD_ID, device="cuda")
        s_in = s_rows
        s_before = s_rows.cpu().numpy()
        if tokens == "oop":
            s_out = torch.full((w.B, W_in + 1 + 5), SENT_TOK, dtype=torch.int32, device="cuda")
        else:
            s_out = s_rows
    if api == "step":
        sd.specdec_step(logits, draft, pad_t, W_in, src, dst, o.tokens, o.n_acc, o.bonus, o.pad_out,
                        o.w_new, o.pos, o.mask, o.workspace, o.dev_status, s_in=s_in, s_out=s_out, pad_id=PAD_ID)
    else:
        sd.specdec_verify_greedy(logits, draft, pad_t, W_in, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                                 o.workspace, o.dev_status)
        sd.specdec_realign_kv(src, dst, w.k, W_in, pad_t, o.n_acc, o.w_new, o.dev_status)
        sd.specdec_build_posmask(o.pad_out, o.w_new, w.k, o.pos, o.mask, o.dev_status)
        if tokens is not None:
            sd.specdec_realign_tokens(s_in, s_out, o.tokens, pad_t, o.n_acc, o.w_new, W_in, PAD_ID, o.dev_status)
    torch.cuda.synchronize()
    out = dict(tokens=o.tokens.cpu().numpy(), n_acc=o.n_acc.cpu().numpy(), bonus=o.bonus.cpu().numpy(),
               pad_out=o.pad_out.cpu().numpy(), w_new=int(o.w_new.cpu()[0]), pos=o.pos.cpu().numpy(),
               mask=o.mask.cpu().numpy(), dev_status=int(o.dev_status.cpu()[0]))
    r = StepResult(w, W_in, cap, np.asarray(pad_in, np.int32), logits, draft, before, dst, out, pm_cap,
                   variant=variant)
    if tokens is not None:
        r.extra.update(s_before=s_before, s_out=s_out.cpu().numpy(), s_out_dev=s_out, tokens=tokens)
    return r


def check_tokens_vs_oracle(r: StepResult, v):
    """The token row against the oracle; out of place, columns beyond w_new+1
    stay untouched."""
    if "s_before" not in r.extra:
        return
    W = v["w_new"]
    exp = oracle.realign_tokens(r.extra["s_before"], v["tokens"], r.pad_in, v["n_acc"], W, r.W_in, PAD_ID)
    got = r.extra["s_out"]
    assert np.array_equal(got[:, :W + 1], exp[:, :W + 1]), "token row differs from the oracle"
    if r.extra["tokens"] == "oop":
        assert np.all(got[:, W + 1:] == SENT_TOK), "token row written beyond w_new + 1"


def check_verify_vs_oracle(r: StepResult):
    w = r.w
    v = oracle.verify(r.logits.cpu(), w.logit_dtype, r.draft.cpu().numpy(), r.pad_in, r.W_in)
    o = r.out
    assert o["dev_status"] == 0, f"device flagged {o['dev_status']:#x}"
    assert np.array_equal(o["tokens"], v["tokens"]), "tokens differ from the oracle"
    assert np.array_equal(o["n_acc"], v["n_acc"]), "accepted counts differ from the oracle"
    assert np.array_equal(o["bonus"], v["bonus"]), "bonus tokens differ from the oracle"
    assert np.array_equal(o["pad_out"], v["pad_out"]), "new paddings differ from the oracle"
    assert o["w_new"] == v["w_new"], "new width differs from the oracle"
    checker.check_geometry(r.pad_in, o["n_acc"], o["pad_out"], o["w_new"], r.W_in, w.k)
    return v


def check_posmask_vs_oracle(r: StepResult, v):
    k = r.w.k
    width = v["w_new"] + k + 1
    pos, mask = oracle.posmask(v["pad_out"], v["w_new"], k, r.pm_cap)
    assert np.array_equal(r.out["pos"][:, :width], pos[:, :width]), "position ids differ from the oracle"
    assert np.array_equal(r.out["mask"][:, :width], mask[:, :width]), "mask differs from the oracle"
    assert np.all(r.out["pos"][:, width:] == SENT_POS), "position ids written beyond w_new+k+1"
    assert np.all(r.out["mask"][:, width:] == SENT_MASK), "mask written beyond w_new+k+1"
    checker.check_posmask(r.out["pos"], r.out["mask"], r.out["pad_out"], r.out["w_new"], k)


def check_kv_full_vs_oracle(r: StepResult, v):
    """Element-by-element comparison of the whole cache (small shapes)."""
    src = bits(r.src)
    dst0 = np.full(src.shape[:4] + (r.dst.shape[4], src.shape[5]), SENT_KV, np.uint16)
    exp = oracle.realign_kv(src, r.w.k, r.W_in, r.pad_in, v["n_acc"], v["w_new"], dst=dst0)
    got = bits(r.dst)
    W = v["w_new"]
    assert np.array_equal(got[..., :W, :], exp[..., :W, :]), _first_diff(got[..., :W, :], exp[..., :W, :])
    return got, exp


def _first_diff(a, b):
    idx = np.argwhere(a != b)
    if idx.size == 0:
        return "equal"
    i = tuple(idx[0])
    return f"first KV difference at {i}: got {a[i]:#06x} want {b[i]:#06x} ({len(idx)} elements differ)"


def check_relocation_on_device(r: StepResult, pad_out, n_acc, w_new):
    """Full-size property check with torch on the device, for every row: pad
    columns [0, pad_out) are +0.0 and content columns [pad_out, w_new) equal
    the kept source columns [pad_in, pad_in + len) bit for bit."""
    L0 = r.W_in - (r.w.k + 1)
    for i in range(r.w.B):
        p, po = int(r.pad_in[i]), int(pad_out[i])
        ln = (L0 - p) + int(n_acc[i]) + 1
        assert po + ln == w_new
        got = i16(r.dst[:, :, i, :, :w_new, :])
        if po:
            assert bool((got[:, :, :, :po, :] == 0).all()), f"row {i}: pads not +0.0"
        want = i16(r.src[:, :, i, :, p:p + ln, :])
        assert torch.equal(got[:, :, :, po:, :], want), f"row {i}: content differs from the kept source columns"


def sample_spans(w: wl.Workload, n_extra: int = 12, seed: int = 0):
    """(layer, row, head) triples covering every row, the first and last span
    and random extras; both K and V of each are compared."""
    rng = np.random.default_rng(seed + 1000)
    spans = {(0, 0, 0), (w.L - 1, w.B - 1, w.H - 1)}
    for b in range(w.B):
        spans.add((int(rng.integers(w.L)), b, int(rng.integers(w.H))))
    for _ in range(n_extra):
        spans.add((int(rng.integers(w.L)), int(rng.integers(w.B)), int(rng.integers(w.H))))
    return sorted(spans)


def host_spans(kv: torch.Tensor, spans, ncols):
    return {s: bits(kv[s[0], :, s[1], s[2], :ncols, :]) for s in spans}


def check_spans_vs_oracle(w, spans, src_spans, dst_spans, pad_in, v, W_in):
    for s in spans:
        l, b, h = s
        src = src_spans[s].reshape(1, 2, 1, 1, W_in, w.D)
        exp = oracle.realign_kv(src, w.k, W_in, pad_in[b:b + 1], v["n_acc"][b:b + 1], v["w_new"])
        got = dst_spans[s]
        W = v["w_new"]
        e = exp.reshape(2, W_in, w.D)[:, :W]
        assert np.array_equal(got[:, :W], e), f"span {s}: " + _first_diff(got[:, :W], e)


class HipBackend:
    """Every step of the method through the library's C ABI, on device
    tensors: the GPU counterpart of ``tests.exspec_loop.OracleBackend``.
    Pool and batch caches are bf16 tensors; token rows, lengths and slots are
    int32 tensors.  ``writeback`` picks the write-back mode."""

    def __init__(self, writeback: int | None = None, device="cuda"):
        from paper_2510_22876_amd import specdec as sd
        self.sd = sd
        self.dev = device
        self.writeback = sd.WRITEBACK_FULL if writeback is None else writeback
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def to_host(self, x):
        if isinstance(x, torch.Tensor):
            if x.dtype == torch.bfloat16:
                return bits(x)
            return x.cpu().numpy()
        return x

    def from_host(self, x):
        if isinstance(x, torch.Tensor):
            return x.to(self.dev)
        x = np.asarray(x)
        if x.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(self.dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(x)).to(self.dev)

    def check_status(self):
        st = int(self.status.cpu()[0])
        assert st == 0, f"device flagged {st:#x}"

    def gather(self, pool, pool_tok, lens, slots, Lb, batch_cap, btok_stride, pad_id):
        L, _, N, H, cap, D = pool.shape
        B = int(slots.numel())
        batch = torch.full((L, 2, B, H, batch_cap, D), SENT_KV, dtype=torch.int16, device=self.dev).view(torch.bfloat16)
        btok = torch.zeros((B, btok_stride), dtype=torch.int32, device=self.dev)
        pads = torch.full((B,), -99, dtype=torch.int32, device=self.dev)
        self.sd.specdec_gather_batch(pool, pool_tok, lens, slots, Lb, batch, pads, batch_tok=btok, pad_id=pad_id,
                                     dev_status=self.status)
        self.check_status()
        return batch, btok, pads

    def posmask(self, pads, width, k, pm_cap):
        B = int(pads.numel())
        pos = torch.full((B, pm_cap), SENT_POS, dtype=torch.int64, device=self.dev)
        mask = torch.full((B, pm_cap), SENT_MASK, dtype=torch.uint8, device=self.dev)
        w = torch.tensor([width], dtype=torch.int32, device=self.dev)
        self.sd.specdec_build_posmask(pads, w, k, pos, mask, self.status)
        self.check_status()
        return pos, mask

    def write_window(self, batch, row, col, entries):
        e = torch.from_numpy(np.ascontiguousarray(entries).view(np.int16)).to(self.dev)
        batch.view(torch.int16)[:, :, row, :, col: col + entries.shape[3], :] = e

    def verify(self, logits, draft, pads, W_in):
        B, kp1, V = logits.shape
        o = self.sd.StepBuffers(B, kp1 - 1, V, W_in + kp1, self.dev)
        self.sd.specdec_verify_greedy(logits, draft, pads, W_in, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                                      o.workspace, self.status)
        self.check_status()
        return dict(tokens=o.tokens, n_acc=o.n_acc, bonus=o.bonus, pad_out=o.pad_out, w_new=o.w_new)

    def rollback(self, tokens, n_acc, pads, W_in):
        B = int(n_acc.numel())
        i32 = dict(dtype=torch.int32, device=self.dev)
        out = dict(n_acc=torch.empty(B, **i32), bonus=torch.empty(B, **i32), pad_out=torch.empty(B, **i32),
                   w_new=torch.empty(1, **i32))
        self.sd.specdec_rollback(tokens, n_acc, pads, W_in, out["n_acc"], out["bonus"], out["pad_out"], out["w_new"],
                                 self.status)
        self.check_status()
        return out

    def scatter(self, batch, pads, tokens, n_acc, slots, Lb, pool, pool_tok, lens, batch_tok):
        self.sd.specdec_scatter_accepted(batch, pads, tokens, n_acc, slots, Lb, pool, pool_tok, lens,
                                         batch_tok=batch_tok, mode=self.writeback, dev_status=self.status)
        self.check_status()

    def realign(self, kv, k, W_in, pads, n_acc, w_new, tokens, s, pad_id):
        out = torch.zeros_like(kv)
        self.sd.specdec_realign_kv(kv, out, k, W_in, pads, n_acc, w_new, self.status)
        s_out = torch.full_like(s, SENT_TOK)
        self.sd.specdec_realign_tokens(s, s_out, tokens, pads, n_acc, w_new, W_in, pad_id, self.status)
        self.check_status()
        return out, s_out
