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
* a replay of every row alone at batch size 1 through the same accept rule;
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


# ---- EXSpec: batch gather, write-back, scheduling (Alg. 2) --------------------------------

def _pool(rng, N, L, H, D, cap, lens, tok_stride):
    """A pool with random entries on [0, len) and garbage (0xFFFF) beyond."""
    pool = np.full((L, 2, N, H, cap, D), 0xFFFF, np.uint16)
    tok = np.full((N, tok_stride), -9, np.int32)
    for s in range(N):
        n = int(lens[s])
        pool[:, :, s, :, :n, :] = rng.integers(1, 0x7F00, size=(L, 2, H, n, D), dtype=np.uint16)
        tok[s, : n + 1] = rng.integers(0, 1000, size=n + 1)
    return pool, tok


def pin_gather_list_model(o=None):
    """Each batch row, read as a list of columns, is the slot's own list of
    cached entries after Lb - len zero columns; its token row is the slot's
    tokens after Lb - len pad ids (checked per element, any width Lb >= the
    longest row, slots in any order, repeated lengths, empty sequences)."""
    rng = np.random.default_rng(21)
    for trial in range(12):
        N = int(rng.integers(1, 9))
        L, H, D = int(rng.integers(1, 3)), int(rng.integers(1, 3)), int(rng.choice([1, 8]))
        cap = 24
        lens = rng.integers(0, cap + 1, size=N).astype(np.int32)
        if trial % 3 == 0:
            lens[:] = lens[0]
        pool, tok = _pool(rng, N, L, H, D, cap, lens, cap + 3)
        B = int(rng.integers(1, N + 1))
        slots = rng.permutation(N)[:B].astype(np.int32)
        Lb = int(lens[slots].max()) + int(rng.integers(0, 3))
        bcap = Lb + int(rng.integers(0, 4))
        bstride = Lb + 1 + int(rng.integers(0, 3))
        out = (np.full((L, 2, B, H, bcap, D), 0xABCD, np.uint16), np.full((B, bstride), -77, np.int32))
        batch, btok, pads = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bstride, -5, out=out, oracle=o)
        for i, s in enumerate(slots):
            n = int(lens[s])
            seq = [pool[:, :, s, :, j, :] for j in range(n)]
            rows = [batch[:, :, i, :, j, :] for j in range(Lb)]
            p = Lb - len(seq)
            assert pads[i] == p
            assert all(not r.any() for r in rows[:p]), "padding columns must be +0.0"
            assert all(np.array_equal(a, b) for a, b in zip(rows[p:], seq))
            assert np.all(batch[:, :, i, :, Lb:, :] == 0xABCD), "columns beyond the width are not written"
            assert list(btok[i, : Lb + 1]) == [-5] * p + list(tok[s, : n + 1])
            assert np.all(btok[i, Lb + 1:] == -77)


def pin_gather_same_length_is_concat(o=None):
    """Same-length rows (Section 3.2): the batch is the plain concatenation of
    the slots' caches along the batch axis, with no padding."""
    rng = np.random.default_rng(22)
    N, L, H, D, cap = 7, 2, 3, 8, 19
    lens = np.full(N, 13, np.int32)
    pool, tok = _pool(rng, N, L, H, D, cap, lens, cap + 2)
    slots = np.array([5, 0, 3, 6], np.int32)
    batch, btok, pads = oracle.gather_batch(pool, tok, lens, slots, 13, 13, 14, -1, oracle=o)
    assert not pads.any()
    want = np.concatenate([pool[:, :, s: s + 1, :, :13, :] for s in slots], axis=2)
    assert np.array_equal(batch, want)
    assert np.array_equal(btok, tok[slots, :14])


def pin_regroup_equals_realign(o=None):
    """Write-back followed by a new gather of the same rows at the new width is
    the EqSpec realignment of the batch (both unpad the rows, append the
    accepted entries and repad to the longest row): two independent routes to
    Section 3.1's unpad-append-repad must agree, also on the token rows."""
    rng = np.random.default_rng(23)
    for trial in range(10):
        N, L, H, D, k = 9, 1, 2, 4, int(rng.integers(0, 5))
        cap = 40
        lens = rng.integers(0, 20, size=N).astype(np.int32)
        pool, tok = _pool(rng, N, L, H, D, cap, lens, cap + 2)
        B = int(rng.integers(1, N + 1))
        slots = rng.permutation(N)[:B].astype(np.int32)
        Lb = int(lens[slots].max())
        bcap = Lb + k + 1
        batch, btok, pads = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bcap + 1, -4, oracle=o)
        # the verify window: fresh entries for [pending, d_1..d_k]
        batch[..., Lb:, :] = rng.integers(1, 0x7F00, size=batch[..., Lb:, :].shape, dtype=np.uint16)
        accepts = rng.integers(0, k + 1, size=B)
        v = _verify_from_accepts(pads, accepts, k, Lb + k + 1, o=o)
        eq = oracle.realign_kv(batch, k, Lb + k + 1, pads, v["n_acc"], v["w_new"], oracle=o)
        eq_tok = oracle.realign_tokens(btok, v["tokens"], pads, v["n_acc"], v["w_new"], Lb + k + 1, -4, oracle=o)
        lens2 = lens.copy()
        oracle.scatter_accepted(batch, pads, v["tokens"], v["n_acc"], slots, Lb, pool, tok, lens2, oracle=o)
        assert np.array_equal(lens2[slots], lens[slots] + v["n_acc"] + 1)
        others = np.setdiff1d(np.arange(N), slots)
        assert np.array_equal(lens2[others], lens[others])
        batch2, btok2, pads2 = oracle.gather_batch(pool, tok, lens2, slots, v["w_new"], v["w_new"], v["w_new"] + 1,
                                                   -4, oracle=o)
        assert np.array_equal(pads2, v["pad_out"])
        assert np.array_equal(batch2, eq[..., : v["w_new"], :])
        assert np.array_equal(btok2, eq_tok[:, : v["w_new"] + 1])


def pin_scatter_appends_to_batch_row(o=None):
    """With the batch token row given, write-back also appends the accepted
    drafts and the bonus to it (Alg. 1's S <- S + A + B): a kept batch then
    equals a new gather of its rows, and with uniform acceptance it equals
    EqSpec's realigned batch at zero offsets (Corollary B.4)."""
    rng = np.random.default_rng(24)
    N, L, H, D, k = 6, 1, 1, 8, 3
    cap = 32
    lens = np.array([10, 4, 10, 7, 10, 1], np.int32)
    pool, tok = _pool(rng, N, L, H, D, cap, lens, cap + 2)
    slots = np.array([0, 2, 4, 1], np.int32)
    Lb = 10
    bcap = Lb + k + 1
    batch, btok, pads = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bcap + 1, -1, oracle=o)
    batch[..., Lb:, :] = rng.integers(1, 0x7F00, size=batch[..., Lb:, :].shape, dtype=np.uint16)
    v = _verify_from_accepts(pads, [2] * 4, k, Lb + k + 1, o=o)
    assert np.array_equal(v["pad_out"], pads)                 # Corollary B.4
    oracle.scatter_accepted(batch, pads, v["tokens"], v["n_acc"], slots, Lb, pool, tok, lens, batch_tok=btok,
                            oracle=o)
    w = v["w_new"]
    assert w == Lb + 3
    again, again_tok, again_pads = oracle.gather_batch(pool, tok, lens, slots, w, w, w + 1, -1, oracle=o)
    assert np.array_equal(again_pads, pads)
    assert np.array_equal(batch[..., :w, :], again)
    assert np.array_equal(btok[:, : w + 1], again_tok)


def _toy_setup(seed, N, V=61, equal_groups=3, lo=3, hi=20):
    from tests.toy_model import ToyModel
    from tests import exspec_loop as el
    rng = np.random.default_rng(seed)
    model = ToyModel(V=V, n_layers=1, H=2, D=4, accept=0.7, salt=seed)
    prompts = el.random_prompts(rng, N, lo, hi, V, equal_groups=equal_groups)
    return model, prompts


def pin_exspec_output_equivalence(o=None):
    """Corollary B.2 for Algorithm 2: an EXSpec loop over a pool (gather,
    verify, write-back, scheduling with lazy realignment and same-length
    grouping) generates, for every sequence, exactly what sequential greedy
    decoding generates, and every slot ends caching its own tokens' entries.
    The toy model turns any cache, mask or position-id error into a changed
    token."""
    from oracle.exspec import SequencePool
    from tests import exspec_loop as el
    for seed, (N, W, B, k, groups) in enumerate([(12, 8, 4, 3, 3), (9, 5, 3, 2, 0), (10, 10, 4, 4, 1)]):
        model, prompts = _toy_setup(seed, N, equal_groups=groups)
        max_new = 12
        sched = SequencePool([len(p) - 1 for p in prompts], window=W, batch=B, max_new=max_new)
        res = el.run_exspec(el.OracleBackend(), model, prompts, sched, k=k, max_new=max_new)
        el.check_equivalence(model, prompts, res, max_new)
        el.check_pool_cache(model, prompts, res)
        assert any(t[2] for t in res.trace) or groups == 0
        assert any(not t[3] for t in res.trace) or groups == 1


def pin_eqspec_output_equivalence(o=None):
    """Corollary B.2 for Algorithm 1: fixed batches realigned after every
    round (cache, token row, positions and mask) generate what sequential
    greedy decoding generates."""
    from tests import exspec_loop as el
    for seed, (N, B, k) in enumerate([(8, 4, 3), (5, 5, 5), (3, 2, 1)]):
        model, prompts = _toy_setup(100 + seed, N, equal_groups=0, lo=2, hi=25)
        res = el.run_eqspec(el.OracleBackend(), model, prompts, B, k, 10)
        el.check_equivalence(model, prompts, res, 10)


def pin_scheduler_properties(o=None):
    """Alg. 2's structure on scheduling traces driven by random acceptance: the
    window holds the first W active sequences, a batch draws min(B, |window|)
    distinct members of it, same-length batches need no padding, a batch is
    kept only after a round whose offsets were all zero (uniform acceptance,
    Corollary B.4), a same-length group is taken whenever the window holds
    B sequences of one length, and every sequence completes."""
    from oracle.exspec import SequencePool
    rng = np.random.default_rng(25)
    for trial in range(30):
        N = int(rng.integers(1, 25))
        W = int(rng.integers(1, 12))
        B = int(rng.integers(1, W + 1))
        k = int(rng.integers(0, 5))
        max_new = int(rng.integers(1, 20))
        lens0 = rng.integers(0, 6 if trial % 2 else 30, size=N)
        sp = SequencePool(list(lens0), window=W, batch=B, max_new=max_new)
        order = sorted(range(N), key=lambda s: (lens0[s], s))
        assert sp.order == order
        prev_uniform = None
        for _ in range(4 * N * (max_new + 1) + 1):
            active = [s for s in order if sp.active[s]]
            b = sp.next_batch()
            if b is None:
                assert not active
                break
            win = active[:W]
            assert len(b.slots) == min(B, len(win)) and len(set(b.slots)) == len(b.slots)
            assert set(b.slots) <= set(win)
            assert b.lens == [sp.len[s] for s in b.slots] and b.width == max(b.lens)
            assert b.same_length == (len(set(b.lens)) == 1)
            if b.reuse:
                assert prev_uniform is not None and prev_uniform == b.slots
            else:
                counts = {}
                for s in win:
                    counts[sp.len[s]] = counts.get(sp.len[s], 0) + 1
                if max(counts.values()) >= len(b.slots):
                    assert b.same_length
                else:
                    assert b.slots == win[: len(b.slots)]
            n_acc = rng.integers(0, k + 1, size=len(b.slots)) if rng.random() < 0.6 else \
                np.full(len(b.slots), int(rng.integers(0, k + 1)))
            before = [sp.len[s] for s in b.slots]
            sp.commit(b, n_acc, [[1] * (int(a) + 1) for a in n_acc])
            assert [sp.len[s] for s in b.slots] == [x + int(a) + 1 for x, a in zip(before, n_acc)]
            prev_uniform = list(b.slots) if len(set(int(a) for a in n_acc)) == 1 and \
                all(sp.active[s] for s in b.slots) else None
        assert b is None and not sp.has_active(), "the schedule did not finish"
        assert all(max_new <= g <= max_new + k for g in sp.generated)


def pin_scheduler_grouping_rate(o=None):
    """Section 3.2: with prompt-length sorting and similar lengths, grouping
    approaches unity.  Equal prompt lengths with uniform acceptance: every
    round runs on a same-length batch, and every round after a batch's first
    keeps it (no gather)."""
    from oracle.exspec import SequencePool
    sp = SequencePool([17] * 12, window=8, batch=4, max_new=10)
    rounds = []
    for _ in range(100):
        b = sp.next_batch()
        if b is None:
            break
        rounds.append((b.same_length, b.reuse))
        sp.commit(b, [2] * len(b.slots), [[1, 1, 1]] * len(b.slots))
    assert b is None and len(rounds) == 12                  # 3 batches of 4, 4 rounds each
    assert all(s for s, _ in rounds)
    assert sum(1 for _, r in rounds if not r) == 3          # one gather per batch of 4


def pin_scheduler_bucket_golden(o=None):
    """Alg. 2's GetBatch grouping on hand-derived windows
    (``tests/golden/sched_bucket_choice.txt``): the oldest window member's
    length bucket when it holds b = min(B, |window|) members, else the largest
    bucket holding b (between equal sizes, the shorter length), else the first
    b window members; the batch's lengths, width and flags follow from the
    chosen slots."""
    from oracle.exspec import SequencePool
    g = _read_golden("sched_bucket_choice.txt")
    cases = sorted({key.split("_", 1)[0] for key in g})
    assert len(cases) == 7, cases
    for c in cases:
        lens0 = g[f"{c}_lens"]
        sp = SequencePool(lens0, window=g[f"{c}_window"][0], batch=g[f"{c}_batch"][0], max_new=1,
                          sort_by_length=False)
        b = sp.next_batch()
        assert b is not None and b.slots == g[f"{c}_slots"], (c, b.slots if b else None)
        lens = [lens0[s] for s in b.slots]
        assert b.lens == lens and b.width == max(lens) and not b.reuse, c
        assert b.same_length == (len(set(lens)) == 1), c


# ---- stochastic verification (T > 0): speculative sampling ---------------------------------------

def _softmax64(x, T):
    z = (np.asarray(x, np.float64) - np.max(x, axis=-1, keepdims=True)) / T
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def pin_sample_preserves_target_distribution(o=None):
    """The guarantee that makes T > 0 decoding output-equivalent: with the draft
    x ~ q_0, the first emitted token is distributed as p_0, and after an
    acceptance the next token as p_1.  Measured exactly by integrating the
    oracle's decisions over a midpoint grid of the two uniforms (error at most
    1/Na + 2/Ns per outcome), for every draft token of a small vocabulary."""
    rng = np.random.default_rng(31)
    V, Na, Ns = 5, 300, 300
    for trial, T in enumerate((0.7, 1.6)):
        tl = rng.normal(0, 1.5, size=(2, V)).astype(np.float32)      # target rows 0 and 1
        dl = rng.normal(0, 1.5, size=(1, V)).astype(np.float32)      # draft row 0
        p0, p1 = _softmax64(tl[0], T), _softmax64(tl[1], T)
        q0 = _softmax64(dl[0], T)
        ua = (np.arange(Na) + 0.5) / Na
        us = (np.arange(Ns) + 0.5) / Ns
        B = V * Na * Ns
        x0 = np.repeat(np.arange(V), Na * Ns).astype(np.int32)
        UA = np.tile(np.repeat(ua, Ns), V).astype(np.float32)
        US = np.tile(us, V * Na).astype(np.float32)
        logits = np.broadcast_to(tl, (B, 2, V))
        dlog = np.broadcast_to(dl, (B, 1, V))
        v = oracle.verify_sample(logits, dlog, "f32", x0.reshape(B, 1), np.zeros(B, np.int32), UA.reshape(B, 1), US,
                                 T, 2, oracle=o)
        first = v["tokens"][:, 0]
        got = np.zeros(V)
        for x in range(V):
            sel = x0 == x
            got += q0[x] * np.bincount(first[sel], minlength=V)[:V] / sel.sum()
        tol = 1.0 / Na + 2.0 / Ns + 1e-9
        assert np.max(np.abs(got - p0)) <= tol, (trial, got, p0)
        acc = v["n_acc"] == 1
        assert np.array_equal(first[acc], x0[acc]) and np.all(first[~acc] != -1)
        # the bonus after an acceptance follows p_1 (over the sampling uniform alone)
        sel = acc & (x0 == int(np.argmax(np.minimum(1.0, p0 / q0))))
        bon = np.bincount(v["bonus"][sel], minlength=V)[:V] / sel.sum()
        assert np.max(np.abs(bon - p1)) <= 2.0 / Ns + 1e-9, (bon, p1)
        # the acceptance rate of each draft token is min(1, p_0(x) / q_0(x))
        for x in range(V):
            sel = x0 == x
            assert abs(acc[sel].mean() - min(1.0, p0[x] / q0[x])) <= 1.0 / Na + 1e-9


def pin_sample_special_cases(o=None):
    """q = p accepts every draft and samples the bonus from p_k by inversion;
    T -> 0 with a clear maximum reduces to greedy verification (Algorithm 3);
    scaling logits and T together changes nothing; a correction token always
    has p_r > q_r; I1 and Eq. (1)-(2) hold."""
    rng = np.random.default_rng(32)
    B, k, V = 6, 3, 40
    tl = rng.normal(0, 2, size=(B, k + 1, V)).astype(np.float32)
    pad = rng.integers(0, 5, size=B).astype(np.int32)
    W_in = 12 + k + 1
    ua = rng.random((B, k)).astype(np.float32)
    us = rng.random(B).astype(np.float32)
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    T = 0.9
    v = oracle.verify_sample(tl, tl[:, :k], "f32", draft, pad, ua, us, T, W_in, oracle=o)
    assert np.all(v["n_acc"] == k)                              # q = p: u * q(x) < q(x) for every u < 1
    for i in range(B):
        cdf = np.cumsum(_softmax64(tl[i, k], T))
        assert v["bonus"][i] == int(np.searchsorted(cdf, float(us[i]) * cdf[-1], side="right"))
        assert list(v["tokens"][i, :k]) == list(draft[i])
    # T -> 0: one-hot distributions; the result is greedy verification's
    for trial in range(4):
        tl = rng.normal(0, 2, size=(B, k + 1, V)).astype(np.float32)
        gl = tl.copy()
        greedy_tok = gl.argmax(-1)
        np.put_along_axis(gl, greedy_tok[..., None], gl.max(-1, keepdims=True) + 8.0, axis=-1)   # 8 above the rest
        acc = rng.integers(0, k + 1, size=B)
        draft = greedy_tok[:, :k].copy()
        for i in range(B):
            if acc[i] < k:
                draft[i, acc[i]] = (draft[i, acc[i]] + 1 + rng.integers(V - 1)) % V
        dl = np.zeros((B, k, V), np.float32)
        dl[np.arange(B)[:, None], np.arange(k)[None, :], draft] = 8.0        # the draft model's own maximum
        vs = oracle.verify_sample(gl.astype(np.float32), dl, "f32", draft.astype(np.int32), pad, ua, us, 0.05, W_in,
                                  oracle=o)
        vg = oracle.verify(gl.astype(np.float32), "f32", draft.astype(np.int32), pad, W_in, oracle=o)
        assert np.array_equal(vs["n_acc"], vg["n_acc"]) and np.array_equal(vs["bonus"], vg["bonus"])
        assert np.array_equal(vs["pad_out"], vg["pad_out"]) and vs["w_new"] == vg["w_new"]
        for i in range(B):
            assert list(vs["tokens"][i, : vs["n_acc"][i] + 1]) == list(vg["tokens"][i, : vg["n_acc"][i] + 1])
    # scale invariance, correction support, geometry
    tl = rng.normal(0, 2, size=(B, k + 1, V)).astype(np.float32)
    dl = rng.normal(0, 2, size=(B, k, V)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    a = oracle.verify_sample(tl, dl, "f32", draft, pad, ua, us, 1.3, W_in, oracle=o)
    b = oracle.verify_sample(tl * 2, dl * 2, "f32", draft, pad, ua, us, 2.6, W_in, oracle=o)
    assert all(np.array_equal(a[x], b[x]) for x in ("tokens", "n_acc", "bonus", "pad_out")) and a["w_new"] == b["w_new"]
    for i in range(B):
        r = int(a["n_acc"][i])
        if r < k:
            t = int(a["bonus"][i])
            assert _softmax64(tl[i, r], 1.3)[t] > _softmax64(dl[i, r], 1.3)[t], "correction outside the residual"
        assert list(a["tokens"][i, :r]) == list(draft[i, :r]) and np.all(a["tokens"][i, r + 1:] == -1)
    from tests import checker
    checker.check_geometry(pad, a["n_acc"], a["pad_out"], a["w_new"], W_in, k)


def pin_sample_widening_exact(o=None):
    """Stochastic verification depends on the logits' values, not only their
    order: a bf16 or f16 logit must enter the softmax exactly as the same
    number held in float32 (every bf16 and f16 value is a float32 value).  The
    oracle on 16-bit logits must therefore decide exactly as the oracle on
    their float32 widenings, made here by numpy's float16 and torch's bfloat16
    conversions.  Rows of normal values at T = 1, rows of subnormals and zeros
    at a temperature of their own scale (where any slip in the subnormal
    scale changes the distribution), and rows of mixed magnitudes with -inf
    entries."""
    rng = np.random.default_rng(33)
    B, k, V = 48, 2, 37
    for dt in ("f16", "bf16"):
        for regime, T in (("normal", 1.0), ("subnormal", 4e-6 if dt == "f16" else 4e-40), ("mixed", 0.8)):
            n = B * (2 * k + 1) * V
            if regime == "normal":
                vals = rng.normal(0, 2, size=n).astype(np.float32)
                bits = (vals.astype(np.float16).view(np.uint16) if dt == "f16" else
                        torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))
            elif regime == "subnormal":
                mant = 0x03FF if dt == "f16" else 0x007F
                bits = (rng.integers(0, mant + 1, size=n) | (rng.integers(0, 2, size=n) << 15)).astype(np.uint16)
            else:
                bits = rng.integers(0, 2 ** 16, size=n).astype(np.uint16)
                expo = (bits >> (10 if dt == "f16" else 7)) & (0x1F if dt == "f16" else 0xFF)
                top = 0x1F if dt == "f16" else 0xFF
                bits = np.where(expo == top, bits & np.uint16(0x83FF if dt == "f16" else 0x807F), bits)  # no inf/NaN
                bits = bits.astype(np.uint16)
                bits[rng.random(n) < 0.1] = 0xFC00 if dt == "f16" else 0xFF80                      # -inf entries
                bits = bits.reshape(-1, V)
                bits[:, 0] = 0x3C00 if dt == "f16" else 0x3F80                                     # a finite maximum per row
                bits = bits.reshape(-1)
            if dt == "f16":
                f32 = bits.view(np.float16).astype(np.float32)
            else:
                f32 = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).float().numpy()
            allb = bits.reshape(B, 2 * k + 1, V)
            allf = f32.reshape(B, 2 * k + 1, V)
            draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
            pad = rng.integers(0, 3, size=B).astype(np.int32)
            ua = rng.random((B, k)).astype(np.float32)
            us = rng.random(B).astype(np.float32)
            W_in = 6 + k + 1
            a = oracle.verify_sample(np.ascontiguousarray(allb[:, : k + 1]), np.ascontiguousarray(allb[:, k + 1:]), dt,
                                     draft, pad, ua, us, T, W_in, oracle=o)
            b = oracle.verify_sample(np.ascontiguousarray(allf[:, : k + 1]), np.ascontiguousarray(allf[:, k + 1:]), "f32",
                                     draft, pad, ua, us, T, W_in, oracle=o)
            for key in ("tokens", "n_acc", "bonus", "pad_out"):
                assert np.array_equal(a[key], b[key]), (dt, regime, key)
            assert a["w_new"] == b["w_new"], (dt, regime)
            # the case is not degenerate: the draws differ from row to row
            assert len(set(int(x) for x in a["bonus"])) > 3, (dt, regime)


# ---- rollback (Family A) and variable-length rollback (Family B) ----------------------------------

def pin_rollback_list_model(o=None):
    """Family A rollback: every row keeps the batch-minimum accepted count m and
    appends tokens[i][0..m]; with Eq. (1)-(2) at a_i = m + 1 every offset is
    equal (zero when the minimum padding is 0, Corollary B.4), so realigning
    the cache moves no entry, and the realigned rows equal a list model that
    keeps c_i + m + 1 entries."""
    rng = np.random.default_rng(41)
    for trial in range(20):
        B, k = int(rng.integers(1, 7)), int(rng.integers(0, 5))
        L = int(rng.integers(k + 1, 20))
        W_in = L + k + 1
        pad = rng.integers(0, L + 1, size=B).astype(np.int32)
        if trial % 2 == 0:
            pad[rng.integers(B)] = 0
        tokens = rng.integers(0, 100, size=(B, k + 1)).astype(np.int32)
        n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
        r = oracle.rollback(tokens, n_acc, pad, W_in, oracle=o)
        m = int(n_acc.min())
        assert np.all(r["n_acc"] == m) and np.array_equal(r["bonus"], tokens[:, m])
        c = L - pad
        assert r["w_new"] == int((c + m + 1).max())
        delta = r["pad_out"] - pad
        assert np.all(delta == delta[0]) and (pad.min() > 0 or delta[0] == 0)
        # the cache: a list model per row, and no move at all when the offsets are zero
        kv = rng.integers(1, 0x7F00, size=(1, 2, B, 2, W_in, 8), dtype=np.uint16)
        for i in range(B):
            kv[:, :, i, :, : pad[i], :] = 0
        out = oracle.realign_kv(kv, k, W_in, pad, r["n_acc"], r["w_new"], oracle=o)
        for i in range(B):
            seq = [kv[:, :, i, :, j, :] for j in range(pad[i], L + m + 1)]
            rows = [out[:, :, i, :, j, :] for j in range(r["pad_out"][i], r["w_new"])]
            assert len(seq) == len(rows) and all(np.array_equal(a, b) for a, b in zip(seq, rows))
        if pad.min() == 0:
            assert np.array_equal(out[..., : r["w_new"], :], kv[..., : r["w_new"], :])


def pin_rollback_output_equivalence(o=None):
    """Family A rollback is correct (Corollary B.2 still holds) but discards
    verified tokens: a rollback decoding loop over the toy model generates what
    sequential greedy decoding generates, in more rounds than dynamic padding."""
    from tests import exspec_loop as el
    for seed, (N, B, k) in enumerate([(6, 3, 4), (4, 4, 3)]):
        model, prompts = _toy_setup(200 + seed, N, equal_groups=0, lo=2, hi=20)
        res = el.run_eqspec(el.OracleBackend(), model, prompts, B, k, 10, rollback=True)
        el.check_equivalence(model, prompts, res, 10)
        dyn = el.run_eqspec(el.OracleBackend(), model, prompts, B, k, 10)
        wasted = sum(sum(a) - len(a) * min(a) for _, _, _, _, a in res.trace)
        assert wasted > 0 and len(res.trace) >= len(dyn.trace)


def _varlen_case(rng, B, k, L, H, D, extra=5):
    c = rng.integers(0, 12, size=B)
    lens = c + k + 1
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T_cap = int(cu[-1]) + extra
    src = rng.integers(1, 0x7F00, size=(L, 2, T_cap, H, D), dtype=np.uint16)
    n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
    return c, cu, src, n_acc, T_cap


def pin_varlen_list_model(o=None):
    """Family B rollback: each sequence, read as a list of rows, keeps its first
    c_i + n_acc_i + 1 rows in order; the offsets are the running sum of the kept
    lengths, each kept row's position id is its index in its sequence, and rows
    beyond the new total are not written."""
    rng = np.random.default_rng(42)
    for trial in range(12):
        B, k = int(rng.integers(1, 6)), int(rng.integers(0, 5))
        c, cu, src, n_acc, T_cap = _varlen_case(rng, B, k, 2, int(rng.integers(1, 3)), 8)
        dst0 = np.full_like(src, 0xABCD)
        out, cu_out, pos = oracle.varlen_rollback(src, cu, n_acc, k, dst=dst0, oracle=o)
        expect_cu = [0]
        for i in range(B):
            seq = [src[:, :, r] for r in range(cu[i], cu[i + 1])][: c[i] + n_acc[i] + 1]
            got = [out[:, :, r] for r in range(cu_out[i], cu_out[i + 1])]
            assert len(seq) == len(got) and all(np.array_equal(a, b) for a, b in zip(seq, got))
            assert list(pos[cu_out[i]: cu_out[i + 1]]) == list(range(len(seq)))
            expect_cu.append(expect_cu[-1] + len(seq))
        assert list(cu_out) == expect_cu
        assert np.all(out[:, :, cu_out[-1]:] == 0xABCD) and np.all(pos[cu_out[-1]:] == -1)


def pin_varlen_equals_padded_realign(o=None):
    """The two layouts agree (Theorem B.1's relocation): a variable-length
    buffer rolled back, and the same sequences left-padded into a rectangular
    batch (windows at [L, L+k+1)) and realigned by EqSpec's unpad-append-repad,
    hold the same rows for every sequence."""
    rng = np.random.default_rng(43)
    for trial in range(8):
        B, k, H, D = int(rng.integers(1, 6)), int(rng.integers(0, 5)), 2, 8
        c, cu, src, n_acc, T_cap = _varlen_case(rng, B, k, 1, H, D)
        out, cu_out, pos = oracle.varlen_rollback(src, cu, n_acc, k, oracle=o)
        L = int(c.max())
        W_in = L + k + 1
        batch = np.zeros((1, 2, B, H, W_in, D), np.uint16)
        pad = (L - c).astype(np.int32)
        for i in range(B):
            batch[:, :, i, :, pad[i]:, :] = np.moveaxis(src[:, :, cu[i]: cu[i + 1]], 2, 3)
        v = _verify_from_accepts(pad, n_acc, k, W_in, o=o)
        re = oracle.realign_kv(batch, k, W_in, pad, v["n_acc"], v["w_new"], oracle=o)
        for i in range(B):
            a = np.moveaxis(re[:, :, i, :, v["pad_out"][i]: v["w_new"], :], 3, 2)
            b = out[:, :, cu_out[i]: cu_out[i + 1]]
            assert np.array_equal(a, b)


ALL_PINS = [
    pin_argmax_bruteforce, pin_argmax_torch, pin_argmax_specials, pin_widening_pairs,
    pin_verify_planted, pin_verify_alg3_vectorised, pin_width_exhaustive,
    pin_corollary_b3, pin_corollary_b4, pin_realign_replay, pin_realign_tagged_chain,
    pin_posmask_closed_form, pin_golden_worked_example, pin_tokens_replay, pin_tokens_chain,
    pin_gather_list_model, pin_gather_same_length_is_concat, pin_regroup_equals_realign,
    pin_scatter_appends_to_batch_row, pin_exspec_output_equivalence, pin_eqspec_output_equivalence,
    pin_scheduler_properties, pin_scheduler_grouping_rate, pin_scheduler_bucket_golden,
    pin_sample_preserves_target_distribution, pin_sample_special_cases, pin_sample_widening_exact,
    pin_rollback_list_model, pin_rollback_output_equivalence, pin_varlen_list_model,
    pin_varlen_equals_padded_realign,
]
