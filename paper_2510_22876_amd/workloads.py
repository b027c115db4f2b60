"""Seeded synthetic workloads for the greedy verify + KV realign step.

This module only *generates inputs*: prompt lengths, intended acceptance
lengths, target logits with a planted maximum per row, draft tokens built
against that planted maximum, and a left-padded bf16 KV cache.  It holds none
of the step's own arithmetic (no argmax, no prefix scan, no width/offset rule,
no relocation): both the oracle tests and the HIP path draw their inputs from
here, and neither depends on the other.

Every random draw is keyed by ``(seed, stream tag, step)`` so that each tensor
and each chained step has its own sub-stream.  Logits and KV are drawn with
``torch.Generator`` on the device where they will live (the multi-GB caches
are generated on the GPU, in place); tests that need the same bytes on the host
copy them back.  The small integer draws (prompt lengths, acceptance lengths, planted
tokens) use numpy on the host so they are identical everywhere.

The five named workloads stand in for the paper's target/draft model pairs
(Vicuna-7B, Qwen3-8B / GLM-4-9B-class GQA models) and SpecBench-style prompt
mixes, which are not available here; the shapes follow the experimental setup
(five draft tokens per round, greedy decoding).
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

# sub-stream tags
_T_PROMPT, _T_ACCEPT, _T_LOGITS, _T_PLANT, _T_DRAFT, _T_TIES, _T_KV, _T_WINDOW, _T_TOKENS = range(1, 10)

DT_CODE = {"f32": 0, "bf16": 1, "f16": 2}
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


@dataclass(frozen=True)
class Workload:
    """Shape and distribution recipe of one synthetic verify+realign workload."""

    name: str
    B: int                       # batch rows
    k: int                       # draft tokens per round
    V: int                       # vocabulary size
    logit_dtype: str             # "f32" | "bf16" | "f16"
    logit_std: float             # logits ~ N(0, std^2) before planting
    L: int                       # layers
    H: int                       # KV heads
    D: int                       # head dim
    prompt: tuple                # ("uniform", lo, hi) | ("loguniform", lo, hi) | ("fixed", n)
    accept: tuple                # ("uniform",) | ("trunc_geom", p) | ("alternate",) | ("fixed", a)
    W_in: Optional[int] = None   # None: max prompt + k + 1 (the longest row has zero padding)
    tie_frac: float = 0.0        # fraction of logit rows with a planted exact tie at the max
    variants: tuple = ("oop", "inplace")
    steps: int = 1               # chained steps (in-place workloads grow the cache by <= k+1 a step)
    extra_cap: int = 0           # cache columns beyond W_in (room for chained growth)

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def column_bytes(self) -> int:
        """Bytes of one KV column across all layers, K/V and heads: L*2*H*D*2."""
        return self.L * 2 * self.H * self.D * 2

    @property
    def logit_bytes(self) -> int:
        return {"f32": 4, "bf16": 2, "f16": 2}[self.logit_dtype]


WORKLOADS = {
    # Tiny: the oracle finishes in milliseconds.  W_in is fixed at 64, so the
    # minimum left pad is >= 19 and the new width sits below the old one
    # (negative, left shifts occur).
    "tiny": Workload("tiny", B=2, k=4, V=1000, logit_dtype="f32", logit_std=1.0,
                     L=2, H=2, D=16, prompt=("uniform", 8, 40), accept=("uniform",), W_in=64),
    # Vicuna-7B-shaped MHA cache, out-of-place realign (the headline workload).
    "vicuna7b": Workload("vicuna7b", B=8, k=5, V=32000, logit_dtype="bf16", logit_std=2.0,
                         L=32, H=32, D=128, prompt=("uniform", 128, 1024),
                         accept=("trunc_geom", 0.6), variants=("oop",)),
    # Same shapes, in-place realign, 16 chained steps.
    "vicuna7b_chained": Workload("vicuna7b_chained", B=8, k=5, V=32000, logit_dtype="bf16",
                                 logit_std=2.0, L=32, H=32, D=128, prompt=("uniform", 128, 1024),
                                 accept=("trunc_geom", 0.6), variants=("inplace",), steps=16,
                                 extra_cap=16 * 6),
    # GQA 8B-shaped, heavily ragged batch.
    "gqa8b": Workload("gqa8b", B=32, k=7, V=128256, logit_dtype="bf16", logit_std=2.0,
                      L=32, H=8, D=128, prompt=("loguniform", 64, 4096), accept=("uniform",)),
    # Stress: long prompts, planted ties, half all-accept / half all-reject.
    "stress": Workload("stress", B=64, k=4, V=151936, logit_dtype="bf16", logit_std=2.0,
                       L=28, H=4, D=128, prompt=("uniform", 512, 8192), accept=("alternate",),
                       tie_frac=0.05),
}


def _rng(seed: int, tag: int, step: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, tag, step]))


def _torch_seed(seed: int, tag: int, step: int = 0, extra: int = 0) -> int:
    ss = np.random.SeedSequence([seed, tag, step, extra])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def prompt_lengths(w: Workload, seed: int = 0) -> np.ndarray:
    """KV-valid prompt lengths n_i (int64 [B])."""
    r = _rng(seed, _T_PROMPT)
    kind = w.prompt[0]
    if kind == "uniform":
        n = r.integers(w.prompt[1], w.prompt[2] + 1, size=w.B)
    elif kind == "loguniform":
        lo, hi = w.prompt[1], w.prompt[2]
        n = np.floor(np.exp(r.uniform(math.log(lo), math.log(hi + 1), size=w.B))).astype(np.int64)
        n = np.clip(n, lo, hi)
    elif kind == "fixed":
        n = np.full(w.B, w.prompt[1], dtype=np.int64)
    elif kind == "list":
        n = np.asarray(w.prompt[1], dtype=np.int64)
    else:
        raise ValueError(kind)
    return n.astype(np.int64)


def initial_geometry(w: Workload, seed: int = 0):
    """(n, W_in, pad_in, cap): left-padded layout of the first verify round.

    Row i holds n_i KV-valid entries in columns [pad_in[i], W0) and the k+1
    verify-window entries in [W0, W_in), W0 = W_in - (k+1).
    """
    n = prompt_lengths(w, seed)
    W_in = w.W_in if w.W_in is not None else int(n.max()) + w.k + 1
    W0 = W_in - (w.k + 1)
    if n.size and int(n.max()) > W0:
        raise ValueError("prompt longer than the cache width")
    pad_in = (W0 - n).astype(np.int32)
    cap = W_in + w.extra_cap
    return n, W_in, pad_in, cap


def intended_accepts(w: Workload, seed: int = 0, step: int = 0) -> np.ndarray:
    """Number of drafts the generator arranges to match the target, per row."""
    r = _rng(seed, _T_ACCEPT, step)
    kind = w.accept[0]
    if kind == "uniform":
        a = r.integers(0, w.k + 1, size=w.B)
    elif kind == "trunc_geom":
        p = w.accept[1]
        # i.i.d. per-draft acceptance with probability p, truncated at k
        probs = np.array([p ** j * (1 - p) for j in range(w.k)] + [p ** w.k])
        a = r.choice(w.k + 1, size=w.B, p=probs / probs.sum())
    elif kind == "alternate":
        a = np.where(np.arange(w.B) % 2 == 0, w.k, 0)
    elif kind == "fixed":
        a = np.full(w.B, w.accept[1])
    elif kind == "list":
        a = np.asarray(w.accept[1])
    else:
        raise ValueError(kind)
    return a.astype(np.int32)


def logits_and_drafts(w: Workload, seed: int = 0, step: int = 0, device="cpu"):
    """Target logits [B,k+1,V] with one planted maximum per row, plus drafts [B,k].

    Each logit row gets a planted token t whose value is (row max + 1), so it
    is the unique maximum unless a tie is planted: in ``tie_frac`` of the rows
    the same value is also written at a second index t2 (half below t, half
    above, at distances from adjacent to far across the row).  ``intended``
    is the token the drafts are planted against: t, or min(t, t2) for a tie
    row.  Drafts copy ``intended`` for the first ``accepts[i]`` slots, differ
    from it at slot ``accepts[i]``, and are uniform afterwards.

    Returns (logits, draft int32, accepts int32 np, intended int32 np, tie_rows np).
    """
    B, k, V = w.B, w.k, w.V
    R = B * (k + 1)
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(seed, _T_LOGITS, step))
    x = torch.randn((R, V), generator=g, device=device, dtype=torch.float32)
    x.mul_(w.logit_std)
    x = x.to(TORCH_DT[w.logit_dtype])
    rp = _rng(seed, _T_PLANT, step)
    planted = rp.integers(0, V, size=R).astype(np.int64)
    if R:
        m = x.float().amax(dim=1) + 1.0
        val = m.to(x.dtype)
        if not bool((val.float() > x.float().amax(dim=1)).all()):
            raise RuntimeError("planted logit is not strictly above the row")
        idx = torch.as_tensor(planted, device=device).view(R, 1)
        x.scatter_(1, idx, val.view(R, 1))
    intended = planted.copy()
    tie_rows = np.zeros(0, dtype=np.int64)
    if w.tie_frac > 0 and V > 1 and R:
        rt = _rng(seed, _T_TIES, step)
        nt = max(1, int(round(w.tie_frac * R)))
        tie_rows = np.sort(rt.choice(R, size=nt, replace=False))
        t2 = np.empty(nt, dtype=np.int64)
        for j, r in enumerate(tie_rows):
            t = planted[r]
            below = (j % 2 == 0)
            far = (j % 4) >= 2
            if below and t == 0:
                below = False
            if not below and t == V - 1:
                below = True
            room = t if below else V - 1 - t
            d = int(rt.integers(1, room + 1)) if far else int(rt.integers(1, min(room, 16) + 1))
            t2[j] = t - d if below else t + d
        tv = x[torch.as_tensor(tie_rows, device=device), torch.as_tensor(planted[tie_rows], device=device)]
        x[torch.as_tensor(tie_rows, device=device), torch.as_tensor(t2, device=device)] = tv
        intended[tie_rows] = np.minimum(planted[tie_rows], t2)
    accepts = intended_accepts(w, seed, step)
    rd = _rng(seed, _T_DRAFT, step)
    intended2 = intended.reshape(B, k + 1)
    draft = rd.integers(0, V, size=(B, k)).astype(np.int64) if V > 0 else np.zeros((B, k), np.int64)
    for i in range(B):
        a = int(accepts[i])
        draft[i, :a] = intended2[i, :a]
        if a < k:
            u = int(rd.integers(0, max(V - 1, 1)))
            draft[i, a] = (intended2[i, a] + 1 + u) % V if V > 1 else intended2[i, a] + 1
    logits = x.view(B, k + 1, V)
    return (logits, torch.as_tensor(draft.astype(np.int32), device=device),
            accepts, intended2.astype(np.int32), tie_rows)


# ---- KV cache ---------------------------------------------------------------

def _mix32(x: torch.Tensor, v) -> torch.Tensor:
    x = (x ^ v) & 0xFFFFFFFF
    x = (x * 0x045D9F3B) & 0xFFFFFFFF
    x = x ^ (x >> 16)
    x = (x * 0x045D9F3B) & 0xFFFFFFFF
    return x ^ (x >> 16)


def kv_tag(step, l, kv, row, head, pos, d, device="cpu") -> torch.Tensor:
    """16-bit tag of one KV element: a finite, non-zero bf16 bit pattern that
    identifies (producing step, layer, K/V, row, head, logical position, dim).

    All arguments broadcast (int tensors or ints); returns an int16 tensor.
    """
    def t(v):
        return torch.as_tensor(v, dtype=torch.int64, device=device)
    x = t(0x9E3779B9)
    for v in (step + 7, l, kv, row, head, pos, d):
        x = _mix32(x, t(v))
    tag = (x & 0xBFFF) | 0x0080           # exponent in [1, 127]: finite and non-zero
    tag = torch.where(tag >= 0x8000, tag - 0x10000, tag)
    return tag.to(torch.int16)


def make_kv(w: Workload, pad_in: np.ndarray, W_in: int, cap: int, seed: int = 0,
            device="cpu", tagged: bool = False, fill_tail: float | None = None) -> torch.Tensor:
    """Left-padded KV cache bf16 [L][2][B][H][cap][D].

    Columns [pad_in[i], W_in) of row i hold values (the prompt's entries and
    the verify window's k+1 entries); columns [0, pad_in[i]) are +0.0 and
    columns [W_in, cap) are +0.0.  Values are N(0,1) rounded to bf16, or, with
    ``tagged``, the tag of (step 0, l, kv, i, h, logical position, d), with the
    logical position counted from the row's first content column.
    """
    L, B, H, D = w.L, w.B, w.H, w.D
    kvt = torch.zeros((L, 2, B, H, cap, D), dtype=torch.bfloat16, device=device)
    col = torch.arange(cap, device=device)
    for l in range(L):
        for kvi in range(2):
            slab = kvt[l, kvi]                       # [B][H][cap][D]
            if tagged:
                pos = col.view(1, 1, cap, 1) - torch.as_tensor(pad_in, device=device).view(B, 1, 1, 1).long()
                vals = kv_tag(0, l, kvi, torch.arange(B, device=device).view(B, 1, 1, 1),
                              torch.arange(H, device=device).view(1, H, 1, 1), pos,
                              torch.arange(D, device=device).view(1, 1, 1, D), device=device)
                vals = vals.view(torch.bfloat16)
            else:
                g = torch.Generator(device=device)
                g.manual_seed(_torch_seed(seed, _T_KV, 0, l * 2 + kvi))
                vals = torch.randn((B, H, cap, D), generator=g, device=device,
                                   dtype=torch.float32).to(torch.bfloat16)
            live = (col.view(1, cap) >= torch.as_tensor(pad_in, device=device).view(B, 1).long()) & \
                   (col.view(1, cap) < W_in)
            slab.copy_(torch.where(live.view(B, 1, cap, 1), vals, torch.zeros((), dtype=torch.bfloat16, device=device)))
            if fill_tail is not None and cap > W_in:
                slab[:, :, W_in:, :] = fill_tail
    return kvt


def write_window(kvt: torch.Tensor, w: Workload, W0: int, pad: np.ndarray, seed: int, step: int,
                 tagged: bool = False) -> None:
    """Write the k+1 verify-window entries of ``step`` at columns [W0, W0+k+1).

    Window slot r of row i is the entry of logical position (W0 - pad[i]) + r.
    """
    L, B, H, D, k = w.L, w.B, w.H, w.D, w.k
    device = kvt.device
    cols = torch.arange(W0, W0 + k + 1, device=device)
    for l in range(L):
        for kvi in range(2):
            if tagged:
                pos = cols.view(1, 1, k + 1, 1) - torch.as_tensor(pad, device=device).view(B, 1, 1, 1).long()
                vals = kv_tag(step, l, kvi, torch.arange(B, device=device).view(B, 1, 1, 1),
                              torch.arange(H, device=device).view(1, H, 1, 1), pos,
                              torch.arange(D, device=device).view(1, 1, 1, D), device=device)
                vals = vals.view(torch.bfloat16)
            else:
                g = torch.Generator(device=device)
                g.manual_seed(_torch_seed(seed, _T_WINDOW, step, l * 2 + kvi))
                vals = torch.randn((B, H, k + 1, D), generator=g, device=device,
                                   dtype=torch.float32).to(torch.bfloat16)
            kvt[l, kvi, :, :, W0:W0 + k + 1, :] = vals


def make_token_rows(w: Workload, pad_in: np.ndarray, W_in: int, stride: int, seed: int = 0, pad_id: int = -1,
                    device="cpu") -> torch.Tensor:
    """Token row S int32 [B][stride]: row i holds pad_in[i] copies of pad_id,
    then c_i + 1 tokens (its cached tokens and the pending token), L + 1
    columns in all, L = W_in - (k+1); later columns hold pad_id.  Tokens are
    uniform in [0, V)."""
    L = W_in - (w.k + 1)
    r = _rng(seed, _T_TOKENS)
    rows = np.full((w.B, stride), pad_id, dtype=np.int32)
    for i in range(w.B):
        p = int(pad_in[i])
        rows[i, p:L + 1] = r.integers(0, max(w.V, 1), size=L + 1 - p)
    return torch.as_tensor(rows, device=device)


# ---- EXSpec sequence pool ------------------------------------------------------

_T_POOL_LEN, _T_POOL_KV, _T_POOL_TOK, _T_POOL_SLOTS = 20, 21, 22, 23


def pool_lengths(w: Workload, N: int, seed: int = 0) -> np.ndarray:
    """Cached entries of N pooled sequences, drawn from the workload's prompt
    distribution (int32 [N])."""
    return prompt_lengths(w.scaled(B=N), seed + 7919 * _T_POOL_LEN).astype(np.int32)


def make_pool(w: Workload, lens: np.ndarray, cap: int, tok_stride: int, seed: int = 0, device="cpu",
              fill: float = 0.0):
    """Sequence pool of EXSpec: cache bf16 [L][2][N][H][cap][D] whose slot s
    holds lens[s] entries (N(0,1) rounded to bf16) in columns [0, lens[s]) and
    ``fill`` beyond; token rows int32 [N][tok_stride] holding lens[s] + 1
    tokens (uniform in [0, V): the cached tokens and the pending one) and -1
    beyond."""
    lens = np.asarray(lens, np.int64)
    N = lens.size
    L, H, D = w.L, w.H, w.D
    pool = torch.empty((L, 2, N, H, cap, D), dtype=torch.bfloat16, device=device)
    col = torch.arange(cap, device=device)
    live = (col.view(1, cap) < torch.as_tensor(lens, device=device).view(N, 1)).view(N, 1, cap, 1)
    fill_t = torch.full((), fill, dtype=torch.bfloat16, device=device)
    for l in range(L):
        for kvi in range(2):
            g = torch.Generator(device=device)
            g.manual_seed(_torch_seed(seed, _T_POOL_KV, 0, l * 2 + kvi))
            vals = torch.randn((N, H, cap, D), generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
            pool[l, kvi].copy_(torch.where(live, vals, fill_t))
    r = _rng(seed, _T_POOL_TOK)
    tok = np.full((N, tok_stride), -1, dtype=np.int32)
    for s in range(N):
        tok[s, : lens[s] + 1] = r.integers(0, max(w.V, 1), size=int(lens[s]) + 1)
    return pool, torch.as_tensor(tok, device=device)


# ---- stochastic verification inputs ----------------------------------------------

_T_SAMPLE_TARGET, _T_SAMPLE_NOISE, _T_SAMPLE_DRAFT, _T_SAMPLE_U = 30, 31, 32, 33


def sampled_inputs(w: Workload, seed: int = 0, step: int = 0, device="cpu", temperature: float = 1.0,
                   noise: float = 1.0):
    """Inputs of one stochastic verification: target logits [B,k+1,V] ~
    N(0, std^2) and draft logits = the first k target rows + N(0, noise^2)
    (both rounded to the workload's logit dtype), so the draft model is a
    perturbed copy of the target: at T = 1 and noise 1 with std 2, each draft
    is accepted with probability about 0.6 (1 - the total-variation distance
    of the two softmaxes); drafts drawn from the draft distribution q; and the
    uniforms u_accept [B,k], u_sample [B] in [0, 1).  Returns (logits,
    draft_logits, draft int32, u_accept, u_sample)."""
    dt = TORCH_DT[w.logit_dtype]
    B, k, V = w.B, w.k, w.V
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(seed, _T_SAMPLE_TARGET, step))
    target = torch.randn((B, k + 1, V), generator=g, device=device, dtype=torch.float32) * w.logit_std
    g.manual_seed(_torch_seed(seed, _T_SAMPLE_NOISE, step))
    dlog = target[:, :k] + torch.randn((B, k, V), generator=g, device=device, dtype=torch.float32) * noise
    logits, draft_logits = target.to(dt), dlog.to(dt)
    q = torch.softmax(draft_logits.float() / temperature, dim=-1).reshape(B * k, V) if k else None
    g.manual_seed(_torch_seed(seed, _T_SAMPLE_DRAFT, step))
    draft = (torch.multinomial(q, 1, generator=g).reshape(B, k).to(torch.int32) if k
             else torch.zeros((B, 0), dtype=torch.int32, device=device))
    g.manual_seed(_torch_seed(seed, _T_SAMPLE_U, step))
    u = torch.rand((B, k + 1), generator=g, device=device, dtype=torch.float32)
    return logits, draft_logits, draft, u[:, :k].contiguous(), u[:, k].contiguous()
