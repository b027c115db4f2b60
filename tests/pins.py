"""Pins of the oracle: checks against what the paper and mathematics fix.

Each ``pin_*`` function takes an ``oracle.Oracle`` handle (or None for the
default build) and raises AssertionError when the oracle disagrees with
something other than itself:

* brute force (a two-pass "find the max value, then the first index holding
  it" scan in pure Python) and ``torch.argmax`` on the CPU for the argmax;
* exact widening checked through pairwise comparisons made by numpy / torch;
* inputs whose answer is known by construction (planted maxima and drafts);
* Algorithm 3's vectorised form written with numpy;
* I1 and the tight-width characterisation of Eq. (1), exhaustively on tiny
  batches; Corollary B.3 (one sequence) and Corollary B.4 (uniform
  acceptance);
* a replay of every row alone at batch size 1 (the spec brute force);
* tagged KV (the cache clause of I2, Theorem B.1, over 16 chained steps);
* the closed form and structure of I2's position ids;
* a worked example derived by hand under ``tests/golden/``.

The same functions run against deliberately broken builds of the oracle
(``test_oracle_mutants.py``) to show that each plausible mistake is caught.
"""
from __future__ import annotations

import itertools
import math
from pathlib import Path

import numpy as np
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests import checker

GOLDEN = Path(__file__).resolve().parent / "golden"


# ---- helpers -----------------------------------------------------------------

def _brute_argmax(vals):
    """Two-pass reference: NaN first (lowest NaN index), else the lowest index
    holding the maximum value."""
    for i, x in enumerate(vals):
        if math.isnan(x):
            return i
    m = max(vals)
    return min(i for i, x in enumerate(vals) if x == m)


def _as_float_list(t: torch.Tensor):
    return [float(x) for x in t.float().tolist()]


# ---- argmax ------------------------------------------------------------------

def pin_argmax_bruteforce(o=None):
    g = torch.Generator().manual_seed(1234)
    for dt in ("f32", "bf16", "f16"):
        for V in (1, 2, 3, 7, 8, 9, 31, 64, 100):
            for trial in range(12):
                # few distinct values -> many exact ties
                x = torch.randint(-3, 4, (V,), generator=g).float() * 0.5
                if trial % 3 == 1:
                    x = torch.randn(V, generator=g)
                if trial % 4 == 2 and V > 1:
                    x[torch.randint(0, V, (1,), generator=g)] = float("nan")
                if trial == 5:
                    x[:] = 0.0
                    x[::2] = -0.0
                t = x.to(wl.TORCH_DT[dt])
                got = oracle.argmax(t, dt, oracle=o)
                want = _brute_argmax(_as_float_list(t))
                assert got == want, (dt, V, trial, got, want)


def pin_argmax_torch(o=None):
    """torch.argmax documents the first occurrence of the maximum and treats NaN
    as the maximum."""
    g = torch.Generator().manual_seed(99)
    for dt in ("f32", "bf16", "f16"):
        for V in (5, 33, 1000, 4099):
            for trial in range(6):
                x = (torch.randn(V, generator=g) * 2).to(wl.TORCH_DT[dt])
                if trial >= 2:       # planted ties at the max, below and above
                    j = int(torch.randint(0, V, (1,), generator=g))
                    j2 = int(torch.randint(0, V, (1,), generator=g))
                    top = x.float().max() + 1
                    x[j] = top.to(x.dtype)
                    x[j2] = top.to(x.dtype)
                if trial == 4:
                    x[int(torch.randint(0, V, (1,), generator=g))] = float("nan")
                want = int(torch.argmax(x))
                got = oracle.argmax(x, dt, oracle=o)
                assert got == want, (dt, V, trial, got, want)


def pin_argmax_specials(o=None):
    cases = [
        ([-0.0, 0.0], 0), ([0.0, -0.0], 0), ([-1.0, -0.0, 0.0], 1),
        ([1.0, float("nan"), 2.0, float("nan")], 1), ([float("nan"), 5.0], 0),
        ([float("-inf"), float("-inf")], 0), ([1.0, float("inf"), float("inf")], 1),
        ([-5.0, -2.0, -2.0, -7.0], 1), ([3.0], 0),
    ]
    for dt in ("f32", "bf16", "f16"):
        for vals, want in cases:
            t = torch.tensor(vals, dtype=torch.float32).to(wl.TORCH_DT[dt])
            assert oracle.argmax(t, dt, oracle=o) == want, (dt, vals)


def pin_widening_pairs(o=None):
    """argmax over [x, y] is 1 exactly when y > x (or y is the first NaN),
    decided here by numpy's float16 and torch's bfloat16/float32 comparisons
    over random bit patterns, subnormals and infinities included."""
    rng = np.random.default_rng(7)
    n = 3000
    for dt in ("f16", "bf16", "f32"):
        if dt == "f32":
            bits = rng.integers(0, 2 ** 32, size=(n, 2), dtype=np.uint64).astype(np.uint32)
            with np.errstate(invalid="ignore"):
                vals = bits.view(np.float32).astype(np.float64)
            raw = bits.view(np.float32)
        else:
            bits = rng.integers(0, 2 ** 16, size=(n, 2), dtype=np.uint64).astype(np.uint16)
            # bias half of them towards small magnitudes (subnormals, +-0)
            bits[: n // 2] &= np.uint16(0x80FF)
            if dt == "f16":
                vals = bits.view(np.float16).astype(np.float64)
            else:
                vals = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
            raw = bits
        for r in range(n):
            x, y = vals[r]
            if math.isnan(x):
                want = 0
            elif math.isnan(y):
                want = 1
            else:
                want = 1 if y > x else 0
            got = oracle.argmax(raw[r], dt, oracle=o)
            assert got == want, (dt, hex(int(bits[r][0])), hex(int(bits[r][1])), got, want)


# ---- verify ------------------------------------------------------------------

def _small(name, **kw):
    return wl.WORKLOADS[name].scaled(**kw)


SMALL_WORKLOADS = [
    wl.WORKLOADS["tiny"],
    _small("vicuna7b", V=3001, L=2, H=2, D=16, prompt=("uniform", 5, 40)),
    _small("gqa8b", V=2053, L=1, H=2, D=8, prompt=("loguniform", 4, 64)),
    _small("stress", B=24, V=4099, L=1, H=1, D=8, prompt=("uniform", 3, 50), tie_frac=0.25),
    _small("tiny", logit_dtype="f16", logit_std=3.0, V=777),
]


def pin_verify_planted(o=None):
    """The generator plants a unique maximum (or a tie whose lowest index it
    knows) and drafts matching it for a known number of slots."""
    for w in SMALL_WORKLOADS:
        for step in range(3):
            n, W_in, pad_in, cap = wl.initial_geometry(w, seed=step)
            logits, draft, accepts, intended, _ = wl.logits_and_drafts(w, seed=step, step=step)
            v = oracle.verify(logits, w.logit_dtype, draft.numpy(), pad_in, W_in, oracle=o)
            assert np.array_equal(v["tokens"], intended), w.name
            assert np.array_equal(v["n_acc"], accepts), w.name
            assert np.array_equal(v["bonus"], intended[np.arange(w.B), accepts]), w.name


def pin_verify_alg3_vectorised(o=None):
    """Algorithm 3's vectorised mismatch detection in numpy, with its all-match
    case read as 'accept all k drafts'."""
    rng = np.random.default_rng(3)
    for w in SMALL_WORKLOADS:
        n, W_in, pad_in, cap = wl.initial_geometry(w)
        logits, draft, *_ = wl.logits_and_drafts(w, seed=5)
        d = draft.numpy().copy()
        # scramble some drafts so mismatches land anywhere
        flip = rng.random(d.shape) < 0.15
        d[flip] = rng.integers(0, w.V, size=int(flip.sum()))
        pred = np.array([[_brute_argmax(_as_float_list(logits[i, r])) for r in range(w.k + 1)]
                         for i in range(w.B)])
        v = oracle.verify(logits, w.logit_dtype, d, pad_in, W_in, oracle=o)
        assert np.array_equal(v["tokens"], pred)
        matches = pred[:, : w.k] == d
        J = np.argmax(~matches, axis=1) if w.k > 0 else np.zeros(w.B, np.int64)
        all_match = matches.all(axis=1) if w.k > 0 else np.ones(w.B, bool)
        J = np.where(all_match, w.k, J)
        assert np.array_equal(v["n_acc"], J)
        assert np.array_equal(v["bonus"], pred[np.arange(w.B), J])


def _verify_from_accepts(pad_in, accepts, k, W_in, V=16, o=None):
    """Run the oracle's verify on fp32 logits whose row maxima are planted at
    token r+1 and drafts that match for exactly ``accepts[i]`` slots."""
    B = len(pad_in)
    logits = np.zeros((B, k + 1, V), np.float32)
    for i in range(B):
        for r in range(k + 1):
            logits[i, r, (r + 1) % V] = 1.0
    draft = np.zeros((B, k), np.int32)
    for i in range(B):
        for r in range(k):
            draft[i, r] = (r + 1) % V if r < accepts[i] else (r + 2) % V
    return oracle.verify(logits, "f32", draft, np.asarray(pad_in, np.int32), W_in, oracle=o)


def pin_width_exhaustive(o=None):
    """Every accepted-count vector for B <= 3, k <= 3 over several pad patterns
    (including every row padded): I1 holds, no padding is negative, the
    longest row is unpadded (Eq. (1)'s max), and the per-row offset equals
    Eq. (2) in the paper's own variables."""
    for B in (1, 2, 3):
        for k in (0, 1, 2, 3):
            W0 = 6
            W_in = W0 + k + 1
            pads = [p for p in itertools.product(range(0, W0 + 1, 2), repeat=B)][:20]
            pads += [tuple([W0] * B), tuple([1] * B)]
            for pad_in in pads:
                for acc in itertools.product(range(k + 1), repeat=B):
                    v = _verify_from_accepts(pad_in, acc, k, W_in, o=o)
                    assert list(v["n_acc"]) == list(acc)
                    checker.check_geometry(pad_in, v["n_acc"], v["pad_out"], v["w_new"], W_in, k)
                    # Eq. (2) with the paper's L = W0 and a_i = accepted + 1
                    a = np.asarray(acc) + 1
                    delta = (v["w_new"] - W0) - a
                    assert np.array_equal(v["pad_out"] - np.asarray(pad_in), delta)


def pin_corollary_b3(o=None):
    """One sequence with no padding: no shift, and the realigned cache is the
    input cache cut at the new width."""
    w = _small("tiny", B=1, prompt=("fixed", 20), W_in=None)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    assert pad_in[0] == 0
    kv = wl.make_kv(w, pad_in, W_in, cap)
    src = kv.view(torch.int16).numpy().view(np.uint16)
    for a in range(w.k + 1):
        v = _verify_from_accepts(pad_in, [a], w.k, W_in, o=o)
        assert v["pad_out"][0] == 0 and v["w_new"] == 20 + a + 1
        out = oracle.realign_kv(src, w.k, W_in, pad_in, v["n_acc"], v["w_new"],
                                dst=np.full(src.shape, 0xFFFF, np.uint16), oracle=o)
        assert np.array_equal(out[..., : v["w_new"], :], src[..., : v["w_new"], :])


def pin_corollary_b4(o=None):
    """Uniform acceptance with the longest row unpadded: every offset is zero and
    the cache is unchanged on [0, width)."""
    w = _small("tiny", B=4, W_in=None, prompt=("list", [9, 30, 17, 30]))
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    kv = wl.make_kv(w, pad_in, W_in, cap)
    src = kv.view(torch.int16).numpy().view(np.uint16)
    for a in range(w.k + 1):
        v = _verify_from_accepts(pad_in, [a] * w.B, w.k, W_in, o=o)
        assert np.array_equal(v["pad_out"], pad_in)
        out = oracle.realign_kv(src, w.k, W_in, pad_in, v["n_acc"], v["w_new"],
                                dst=np.full(src.shape, 0xFFFF, np.uint16), oracle=o)
        assert np.array_equal(out[..., : v["w_new"], :], src[..., : v["w_new"], :])


# ---- realign -------------------------------------------------------------------

def _replay_row(src_row, pad, W0, n_acc):
    """Batch-size-1 replay of one row (all heads, layers): the sequence alone,
    unpadded, as a Python list of cached columns; the step appends the
    pending token's entry and each accepted draft's entry in order."""
    seq = [src_row[..., j, :] for j in range(pad, W0)]        # its own cache, no padding
    window = [src_row[..., W0 + r, :] for r in range(n_acc + 1)]
    for e in window:                                          # one append per kept token
        seq.append(e)
    return seq


def pin_realign_replay(o=None):
    for w in SMALL_WORKLOADS:
        for seed in range(3):
            n, W_in, pad_in, cap = wl.initial_geometry(w, seed=seed)
            W0 = W_in - (w.k + 1)
            logits, draft, *_ = wl.logits_and_drafts(w, seed=seed)
            kv = wl.make_kv(w, pad_in, W_in, cap, seed=seed)
            src = kv.view(torch.int16).numpy().view(np.uint16)
            v = oracle.verify(logits, w.logit_dtype, draft.numpy(), pad_in, W_in, oracle=o)
            dst = np.full(src.shape, 0xFFFF, np.uint16)
            out = oracle.realign_kv(src, w.k, W_in, pad_in, v["n_acc"], v["w_new"], dst=dst, oracle=o)
            pos, mask = oracle.posmask(v["pad_out"], v["w_new"], w.k, oracle=o)
            for i in range(w.B):
                seq = _replay_row(src[:, :, i], int(pad_in[i]), W0, int(v["n_acc"][i]))
                p = int(v["pad_out"][i])
                assert p + len(seq) == v["w_new"]
                got = out[:, :, i, :, : v["w_new"], :]
                assert np.all(got[..., :p, :] == 0), "pads must be +0.0"
                for j, e in enumerate(seq):
                    assert np.array_equal(got[..., p + j, :], e), (w.name, i, j)
                # position ids of the replayed sequence are 0..len-1
                assert list(pos[i, p: v["w_new"]]) == list(range(len(seq)))


def pin_realign_tagged_chain(o=None):
    """Theorem B.1 by induction over 16 chained steps on tagged KV: after every
    step each content column holds its own position's entry from the step that
    accepted it, pads are zero, and position ids agree with the tags."""
    for w in (wl.WORKLOADS["tiny"].scaled(W_in=None, extra_cap=16 * 5),
              _small("vicuna7b", V=997, L=1, H=2, D=8, prompt=("uniform", 3, 30),
                     extra_cap=16 * 6)):
        n, W_in, pad_in, cap = wl.initial_geometry(w)
        kv = wl.make_kv(w, pad_in, W_in, cap, tagged=True)
        cur = kv.view(torch.int16).numpy().view(np.uint16).copy()
        prod = [np.zeros(int(n[i]), np.int64) for i in range(w.B)]
        pad = pad_in.copy()
        W0 = W_in - (w.k + 1)
        for step in range(16):
            if step > 0:
                t = torch.from_numpy(cur.view(np.int16)).view(torch.bfloat16)
                wl.write_window(t, w, W0, pad, seed=0, step=step, tagged=True)
            Wi = W0 + w.k + 1
            logits, draft, accepts, *_ = wl.logits_and_drafts(w, seed=0, step=step)
            v = oracle.verify(logits, w.logit_dtype, draft.numpy(), pad, Wi, oracle=o)
            checker.check_geometry(pad, v["n_acc"], v["pad_out"], v["w_new"], Wi, w.k)
            nxt = np.full_like(cur, 0xFFFF)
            oracle.realign_kv(cur, w.k, Wi, pad, v["n_acc"], v["w_new"], dst=nxt, oracle=o)
            n_before = W0 - pad
            prod = checker.advance_prod_steps(prod, n_before, v["n_acc"], step)
            checker.check_tagged_kv(nxt, v["pad_out"], v["w_new"], prod)
            pos, mask = oracle.posmask(v["pad_out"], v["w_new"], w.k, oracle=o)
            checker.check_posmask(pos, mask, v["pad_out"], v["w_new"], w.k)
            # columns [w_new, cap) are unspecified after a step; clear them like a fresh cache
            nxt[..., v["w_new"]:, :] = 0
            cur, pad, W0 = nxt, v["pad_out"].copy(), v["w_new"]


# ---- position ids and mask ---------------------------------------------------------

def pin_posmask_closed_form(o=None):
    rng = np.random.default_rng(11)
    for trial in range(40):
        B = int(rng.integers(1, 9))
        k = int(rng.integers(0, 8))
        w_new = int(rng.integers(0, 50))
        pad_out = rng.integers(0, w_new + 1, size=B).astype(np.int32)
        pm_cap = w_new + k + 1 + int(rng.integers(0, 4))
        pos, mask = oracle.posmask(pad_out, w_new, k, pm_cap, oracle=o)
        j = np.arange(w_new + k + 1)
        for i in range(B):
            assert np.array_equal(mask[i, : w_new + k + 1], (j >= pad_out[i]).astype(np.uint8))
            assert np.array_equal(pos[i, : w_new + k + 1], np.maximum(0, j - pad_out[i]))
        checker.check_posmask(pos, mask, pad_out, w_new, k)


# ---- the hand-worked example ---------------------------------------------------------

def _read_golden(name):
    vals = {}
    for line in (GOLDEN / name).read_text().splitlines():
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, _, rest = line.partition("=")
        vals[key.strip()] = [float(x) if ("." in x or "n" in x) else int(x) for x in rest.split()]
    return vals


def pin_golden_worked_example(o=None):
    g = _read_golden("worked_example_b3k2.txt")
    B, k, V, W_in = g["B"][0], g["k"][0], g["V"][0], g["W_in"][0]
    logits = np.asarray(g["logits"], np.float32).reshape(B, k + 1, V)
    draft = np.asarray(g["draft"], np.int32).reshape(B, k)
    pad_in = np.asarray(g["pad_in"], np.int32)
    v = oracle.verify(logits, "f32", draft, pad_in, W_in, oracle=o)
    assert list(v["tokens"].reshape(-1)) == g["tokens"]
    assert list(v["n_acc"]) == g["n_acc"]
    assert list(v["bonus"]) == g["bonus"]
    assert v["w_new"] == g["w_new"][0]
    assert list(v["pad_out"]) == g["pad_out"]
    # KV: one layer, one head, D=1; every source column holds its own column index + 1
    src = np.zeros((1, 2, B, 1, W_in, 1), np.uint16)
    for i in range(B):
        src[:, :, i, 0, pad_in[i]:, 0] = np.arange(pad_in[i], W_in) + 1
    out = oracle.realign_kv(src, k, W_in, pad_in, v["n_acc"], v["w_new"],
                            dst=np.full(src.shape, 0xFFFF, np.uint16), oracle=o)
    for i in range(B):
        assert list(out[0, 0, i, 0, : v["w_new"], 0]) == g[f"kv_row{i}"]
        assert list(out[0, 1, i, 0, : v["w_new"], 0]) == g[f"kv_row{i}"]
    pos, mask = oracle.posmask(v["pad_out"], v["w_new"], k, oracle=o)
    for i in range(B):
        assert list(pos[i]) == g[f"pos_row{i}"]
        assert list(mask[i]) == g[f"mask_row{i}"]
    s_in = np.asarray([g[f"s_in_row{i}"] for i in range(B)], np.int32)
    s_out = oracle.realign_tokens(s_in, v["tokens"], pad_in, v["n_acc"], v["w_new"], W_in, g["pad_id"][0], oracle=o)
    for i in range(B):
        assert list(s_out[i]) == g[f"s_out_row{i}"]


# ---- token row (Alg. 1, phase 3) -------------------------------------------------------

def pin_tokens_replay(o=None):
    """Each row alone: its own tokens (cached + pending) followed by the accepted
    drafts D[i][:n_acc] and the bonus B[i] (Alg. 1's append); the realigned
    row must be that list after pad_out[i] pads, with the same padding as the
    cache (I1 shared by S and the cache)."""
    for w in SMALL_WORKLOADS:
        for seed in range(3):
            n, W_in, pad_in, cap = wl.initial_geometry(w, seed=seed)
            L = W_in - (w.k + 1)
            logits, draft, *_ = wl.logits_and_drafts(w, seed=seed)
            d = draft.numpy()
            v = oracle.verify(logits, w.logit_dtype, d, pad_in, W_in, oracle=o)
            s_in = wl.make_token_rows(w, pad_in, W_in, W_in + 2, seed=seed, pad_id=-3).numpy()
            out = oracle.realign_tokens(s_in, v["tokens"], pad_in, v["n_acc"], v["w_new"], W_in, -3, oracle=o)
            assert out.shape[1] == v["w_new"] + 1
            for i in range(w.B):
                seq = list(s_in[i, pad_in[i]:L + 1])
                seq += list(d[i, : v["n_acc"][i]]) + [v["bonus"][i]]
                p = v["w_new"] + 1 - len(seq)
                assert p == v["pad_out"][i], "token row and cache disagree on the padding"
                assert list(out[i, :p]) == [-3] * p
                assert list(out[i, p:]) == seq, (w.name, seed, i)


def pin_tokens_chain(o=None):
    """16 chained steps: the token row, grown by Alg. 1's append each step,
    stays equal to a per-row list model and keeps exactly one more token than
    the cache (the pending token), left-aligned to the same padding."""
    w = _small("vicuna7b", V=997, L=1, H=1, D=8, prompt=("uniform", 3, 30), extra_cap=16 * 6)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    L = W_in - (w.k + 1)
    s = wl.make_token_rows(w, pad_in, W_in, cap + 2, pad_id=-1).numpy()
    model = [list(s[i, pad_in[i]:L + 1]) for i in range(w.B)]
    pad, W0 = pad_in.copy(), L
    for step in range(16):
        Wi = W0 + w.k + 1
        logits, draft, *_ = wl.logits_and_drafts(w, seed=0, step=step)
        d = draft.numpy()
        v = oracle.verify(logits, w.logit_dtype, d, pad, Wi, oracle=o)
        s = oracle.realign_tokens(s, v["tokens"], pad, v["n_acc"], v["w_new"], Wi, -1, out_stride=cap + 2, oracle=o)
        for i in range(w.B):
            model[i] += list(d[i, : v["n_acc"][i]]) + [v["bonus"][i]]
            po = v["pad_out"][i]
            assert list(s[i, po: v["w_new"] + 1]) == model[i]
            assert len(model[i]) == (v["w_new"] - po) + 1     # cache content + the pending token
        pad, W0 = v["pad_out"].copy(), v["w_new"]


ALL_PINS = [
    pin_argmax_bruteforce, pin_argmax_torch, pin_argmax_specials, pin_widening_pairs,
    pin_verify_planted, pin_verify_alg3_vectorised, pin_width_exhaustive,
    pin_corollary_b3, pin_corollary_b4, pin_realign_replay, pin_realign_tagged_chain,
    pin_posmask_closed_form, pin_golden_worked_example, pin_tokens_replay, pin_tokens_chain,
]
