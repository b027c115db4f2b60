"""Invariant checker for one verify+realign step, independent of both the oracle
and the HIP library.

It checks what the paper fixes without recomputing the step the way either
implementation does:

* I1, rectangular alignment (Section 3.1): every row's new padding plus its
  new content length equals the one shared width, no padding is negative, and
  the longest row carries no padding (the width is the tight maximum of
  Eq. (1)).
* I2, position ids (Section 3.1): the first content column has position 0 and
  positions rise by one per content column; pad columns have position 0 and
  mask 0.
* The cache clause of I2 (Theorem B.1): with tagged KV, every content column
  holds the entry produced for its own logical position (and in the step that
  accepted it), pad columns hold +0.0, and no rejected entry survives.
"""
from __future__ import annotations

import numpy as np
import torch

from paper_2510_22876_amd.workloads import kv_tag


class InvariantError(AssertionError):
    pass


def check_geometry(pad_in, n_acc, pad_out, w_new, W_in, k):
    pad_in = np.asarray(pad_in, np.int64)
    n_acc = np.asarray(n_acc, np.int64)
    pad_out = np.asarray(pad_out, np.int64)
    W0 = W_in - (k + 1)
    if np.any(n_acc < 0) or np.any(n_acc > k):
        raise InvariantError(f"accepted counts out of [0,{k}]: {n_acc}")
    new_len = (W0 - pad_in) + n_acc + 1
    if np.any(pad_out + new_len != w_new):
        raise InvariantError(f"I1 broken: pad_out {pad_out} + len {new_len} != width {w_new}")
    if np.any(pad_out < 0):
        raise InvariantError(f"negative padding {pad_out}")
    if pad_out.size and pad_out.min() != 0:
        raise InvariantError(f"width {w_new} is not tight: min padding {pad_out.min()}")


def check_posmask(pos, mask, pad_out, w_new, k):
    pos = np.asarray(pos)
    mask = np.asarray(mask)
    width = w_new + k + 1
    for i, p in enumerate(np.asarray(pad_out)):
        m = mask[i, :width]
        ps = pos[i, :width]
        if np.any(m[:p] != 0) or np.any(m[p:] != 1):
            raise InvariantError(f"row {i}: mask does not switch on at column {p}")
        if np.any(ps[:p] != 0):
            raise InvariantError(f"row {i}: pad columns carry non-zero positions")
        seg = ps[p:]
        if seg.size and (seg[0] != 0 or np.any(np.diff(seg) != 1)):
            raise InvariantError(f"row {i}: content positions are not 0,1,2,...")


def expected_tags(l, kv, row, H, D, w_new, pad_out, prod_step, device="cpu"):
    """bf16 bit patterns [H][w_new][D] that row ``row`` of slab (l, kv) must
    hold: +0.0 on pads, the tag of (producing step, l, kv, row, h, p, d) on
    content column pad_out + p.  Returns numpy uint16 on the CPU, an int16
    tensor on another device."""
    p0 = int(pad_out)
    n = w_new - p0
    out = torch.zeros((H, w_new, D), dtype=torch.int16, device=device)
    if n > 0:
        steps = torch.as_tensor(np.asarray(prod_step[:n]), dtype=torch.int64, device=device).view(1, n, 1)
        tags = kv_tag(steps, l, kv, row, torch.arange(H, device=device).view(H, 1, 1),
                      torch.arange(n, device=device).view(1, n, 1), torch.arange(D, device=device).view(1, 1, D),
                      device=device)
        out[:, p0:, :] = tags
    if device == "cpu":
        return out.numpy().view(np.uint16)
    return out


def check_tagged_kv_device(kv: torch.Tensor, pad_out, w_new, prod_steps):
    """check_tagged_kv for a bf16 cache that stays on its device."""
    L, _, B, H, cap, D = kv.shape
    for l in range(L):
        for k2 in range(2):
            for i in range(B):
                exp = expected_tags(l, k2, i, H, D, w_new, pad_out[i], prod_steps[i], device=kv.device)
                got = kv[l, k2, i, :, :w_new, :].view(torch.int16)
                if not torch.equal(got, exp):
                    bad = (got != exp).nonzero()[0].tolist()
                    raise InvariantError(f"cache clause broken at layer {l} kv {k2} row {i} head/col {bad} "
                                         f"(pad_out {pad_out[i]})")


def check_tagged_kv(kv_bits, pad_out, w_new, prod_steps, layers=None, rows=None):
    """kv_bits: uint16 [L][2][B][H][cap][D] after realign; prod_steps[i] gives the
    producing step of each logical position of row i (length >= new length)."""
    L, _, B, H, cap, D = kv_bits.shape
    layers = range(L) if layers is None else layers
    rows = range(B) if rows is None else rows
    for l in layers:
        for kv in range(2):
            for i in rows:
                exp = expected_tags(l, kv, i, H, D, w_new, pad_out[i], prod_steps[i])
                got = kv_bits[l, kv, i, :, :w_new, :]
                if not np.array_equal(got, exp):
                    bad = np.argwhere(got != exp)[0]
                    raise InvariantError(
                        f"cache clause broken at layer {l} kv {kv} row {i} head {bad[0]} col {bad[1]} "
                        f"(pad_out {pad_out[i]}): got {got[tuple(bad)]:#06x} want {exp[tuple(bad)]:#06x}")


def advance_prod_steps(prod_steps, n_before, n_acc, step):
    """Producing-step bookkeeping: row i had n_before[i] cached entries; this
    step kept n_acc[i]+1 more (the pending token and the accepted drafts)."""
    out = []
    for i, ps in enumerate(prod_steps):
        keep = list(ps[: int(n_before[i])]) + [step] * (int(n_acc[i]) + 1)
        out.append(np.asarray(keep, np.int64))
    return out
