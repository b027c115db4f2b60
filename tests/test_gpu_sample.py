"""GPU parity of stochastic (T > 0) verification (speculative sampling)
through the C ABI against the oracle on the same inputs and uniforms.

The kernels decide integers (accept / reject, the index drawn by inversion)
from fp32 sums over the vocabulary; the oracle takes the same decisions in
fp64.  A decision can therefore differ only where the oracle's margin is
inside the fp32 rounding of those sums.  The bound used (the derivation is
in the design notes): the ratio p(x)/q(x) is within a relative 2e-4 of the
fp64 value, and a cumulative fraction of the sampling weights within an
absolute 2e-4 / m of it, m being the total weight (the residual's mass, 1
for the bonus).  A row must equal the oracle exactly, or, when the oracle's
result changes inside that band, equal the oracle's result at one of the
band's edges.  Rows that needed the band are counted; they must be rare.
"""
import numpy as np
import pytest
import torch

import oracle
from tests import checker
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

DA, DS = 2e-4, 2e-4


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec
    return specdec


TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


def _softmax64(x, T):
    x = np.asarray(x, np.float64)
    z = (x - np.max(x, axis=-1, keepdims=True)) / T
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def _make(rng, B, k, V, dtype, T, std=2.0, mode="sampled", mask_frac=0.0):
    """Target / draft logits (rounded to dtype), drafts drawn from q (mode
    'sampled'), equal to the target's argmax ('greedy'), or uniform ('uniform');
    uniforms in [0, 1)."""
    tl = torch.tensor(rng.normal(0, std, size=(B, k + 1, V)), dtype=TORCH[dtype])
    dl = torch.tensor(rng.normal(0, std, size=(B, k, V)), dtype=TORCH[dtype])
    if mask_frac:
        m = rng.random((B, k + 1, V)) < mask_frac
        m[..., 0] = False                                  # keep a finite maximum
        tl[torch.from_numpy(m)] = float("-inf")
        dl[torch.from_numpy(m[:, :k])] = float("-inf")
    q = _softmax64(dl.float().numpy(), T)
    if mode == "sampled":
        cdf = np.cumsum(q, axis=-1)
        u = rng.random((B, k, 1))
        draft = np.minimum((cdf < u * cdf[..., -1:]).sum(-1), V - 1)
    elif mode == "greedy":
        draft = tl.float().numpy()[:, :k].argmax(-1)
    else:
        draft = rng.integers(0, V, size=(B, k))
    ua = rng.random((B, k)).astype(np.float32)
    us = rng.random(B).astype(np.float32)
    return tl, dl, draft.astype(np.int32), ua, us


def _run_gpu(sd, tl, dl, draft, pad, ua, us, T, W_in):
    B, kp1, V = tl.shape
    k = kp1 - 1
    dev = "cuda"
    i32 = dict(dtype=torch.int32, device=dev)
    out = dict(tokens=torch.full((B, kp1), -99, **i32), n_acc=torch.full((B,), -99, **i32),
               bonus=torch.full((B,), -99, **i32), pad_out=torch.full((B,), -99, **i32),
               w_new=torch.full((1,), -99, **i32))
    st = torch.zeros(1, **i32)
    ws = sd.alloc_sample_workspace(B, k, V, dev)
    ws.fill_(-1)                                           # garbage: the workspace needs no initialisation
    sd.specdec_verify_sample(tl.to(dev), dl.to(dev), torch.as_tensor(draft, device=dev), torch.as_tensor(pad, device=dev),
                             torch.as_tensor(ua, device=dev), torch.as_tensor(us, device=dev), T, W_in, out["tokens"],
                             out["n_acc"], out["bonus"], out["pad_out"], out["w_new"], ws, st)
    torch.cuda.synchronize()
    res = {n: t.cpu().numpy() for n, t in out.items()}
    res["w_new"] = int(res["w_new"][0])
    res["status"] = int(st.cpu()[0])
    return res


def _row(v, i):
    n = int(v["n_acc"][i])
    return n, tuple(int(t) for t in v["tokens"][i, : n + 1])


def check_against_oracle(tl, dl, dtype, draft, pad, ua, us, T, W_in, got):
    """Exact agreement, or agreement with the oracle somewhere in the fp32
    band; returns the number of rows that needed the band.

    The accept tests are decided on u_accept, which the band moves by
    a relative delta_a; the drawn token is the inversion of u_sample, which
    it moves by delta_s / m (m = the mass of the weights sampled from).  For
    a fixed accept outcome the token is non-decreasing in u_sample, so every
    token between the oracle's draws at the two ends of the band is one that
    some u_sample in the band produces."""
    B, kp1, V = tl.shape
    k = kp1 - 1
    args = (tl, dl, dtype, draft, pad)
    nom = oracle.verify_sample(*args, ua, us, T, W_in)
    assert got["status"] == 0, f"device flagged {got['status']:#x}"
    # masses of the weights each row sampled from (residual at the rejected slot, else 1)
    p = _softmax64(tl.float().numpy(), T)
    q = _softmax64(dl.float().numpy(), T)
    banded = 0
    edges = None
    for i in range(B):
        if _row(got, i) == _row(nom, i):
            continue
        if edges is None:
            j = nom["n_acc"]
            mass = np.ones(B)
            rej = j < k
            if k:
                r = np.minimum(j, k - 1)
                mass[rej] = np.maximum(p[np.arange(B), r] - q[np.arange(B), r], 0).sum(-1)[rej]
            ds = DS / np.maximum(mass, 1e-3)
            edges = {}
            for sa in (-1, 0, 1):
                ua2 = np.clip(ua * (1 + sa * DA), 0, np.float32(0.99999994)).astype(np.float32)
                for ss in (-1, 0, 1):
                    us2 = np.clip(us + ss * ds, 0, np.float32(0.99999994)).astype(np.float32)
                    edges[sa, ss] = oracle.verify_sample(*args, ua2, us2, T, W_in)
        n_got, toks = _row(got, i)
        ok = False
        for sa in (-1, 0, 1):
            lo, hi = _row(edges[sa, -1], i), _row(edges[sa, 1], i)
            if lo[0] != n_got or lo[1][:n_got] != toks[:n_got]:
                continue
            ok = lo[1][n_got] <= toks[n_got] <= hi[1][n_got]
            if ok:
                break
        assert ok, f"row {i}: GPU {(n_got, toks)} vs oracle {_row(nom, i)} (outside the fp32 band)"
        banded += 1
    # geometry follows from the accepted counts exactly
    checker.check_geometry(pad, got["n_acc"], got["pad_out"], got["w_new"], W_in, k)
    assert np.all(got["bonus"] == got["tokens"][np.arange(B), got["n_acc"]])
    for i in range(B):
        n = int(got["n_acc"][i])
        assert list(got["tokens"][i, :n]) == list(draft[i, :n]) and np.all(got["tokens"][i, n + 1:] == -1)
        assert 0 <= got["bonus"][i] < V
    return banded


CASES = [
    # B, k, V, dtype, T, mode
    (4, 5, 1000, "f32", 1.0, "sampled"),
    (8, 5, 32000, "bf16", 0.8, "sampled"),
    (16, 7, 4093, "bf16", 1.5, "sampled"),      # ragged vocabulary: unaligned rows
    (3, 4, 7, "f16", 0.5, "uniform"),
    (5, 0, 333, "bf16", 1.0, "sampled"),        # k = 0: only the bonus
    (2, 64, 129, "f32", 2.0, "sampled"),        # k = 64: every lane of wave 0
    (6, 3, 1, "f32", 1.0, "uniform"),           # V = 1
    (64, 4, 151936, "bf16", 0.7, "sampled"),    # stress-shaped vocabulary
    (8, 5, 32000, "bf16", 0.05, "greedy"),      # near-greedy
    (3, 1, 1000000, "f32", 0.9, "sampled"),     # 64 chunks of 8 tiles
    (2, 2, 5000000, "bf16", 1.0, "sampled"),    # 39 tiles per chunk
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}k{}V{}{}T{}{}".format(*c))
@pytest.mark.parametrize("seed", [0, 1])
def test_verify_sample_matches_oracle(sd, case, seed):
    B, k, V, dtype, T, mode = case
    say(f"verify_sample case={case} seed={seed}")
    rng = np.random.default_rng(1000 * seed + V + k)
    tl, dl, draft, ua, us = _make(rng, B, k, V, dtype, T, mode=mode)
    pad = rng.integers(0, 9, size=B).astype(np.int32)
    W_in = 20 + k + 1
    got = _run_gpu(sd, tl, dl, draft, pad, ua, us, T, W_in)
    banded = check_against_oracle(tl, dl, dtype, draft, pad, ua, us, T, W_in, got)
    say(f"  n_acc={got['n_acc'].tolist()[:16]} banded rows={banded}")
    assert banded <= max(1, B // 16)


def test_verify_sample_many_rows_band_is_rare(sd):
    """4096 rows of a small vocabulary: the band is needed for a tiny fraction."""
    rng = np.random.default_rng(9)
    B, k, V, T = 4096, 3, 257, 0.9
    tl, dl, draft, ua, us = _make(rng, B, k, V, "bf16", T)
    pad = np.zeros(B, np.int32)
    got = _run_gpu(sd, tl, dl, draft, pad, ua, us, T, k + 1 + 3)
    banded = check_against_oracle(tl, dl, "bf16", draft, pad, ua, us, T, k + 1 + 3, got)
    say(f"  banded rows {banded} of {B}")
    assert banded <= 8


def test_verify_sample_equal_distributions_accept_all(sd):
    """q = p: every draft is accepted, whatever the uniforms (u < 1)."""
    rng = np.random.default_rng(10)
    B, k, V, T = 32, 6, 5000, 1.1
    tl = torch.tensor(rng.normal(0, 2, size=(B, k + 1, V)), dtype=torch.bfloat16)
    dl = tl[:, :k].clone()
    draft = rng.integers(0, V, size=(B, k)).astype(np.int32)
    ua = np.full((B, k), 0.99999994, np.float32)
    us = rng.random(B).astype(np.float32)
    pad = np.zeros(B, np.int32)
    got = _run_gpu(sd, tl, dl, draft, pad, ua, us, T, k + 1)
    assert np.all(got["n_acc"] == k)
    check_against_oracle(tl, dl, "bf16", draft, pad, ua, us, T, k + 1, got)


def test_verify_sample_masked_and_out_of_range(sd):
    """-inf logits (masked vocabulary entries) have probability 0 and are never
    drawn; draft ids outside [0, V) are rejected."""
    rng = np.random.default_rng(11)
    B, k, V, T = 12, 4, 3000, 1.0
    tl, dl, draft, ua, us = _make(rng, B, k, V, "bf16", T, mask_frac=0.5)
    draft[0, 0] = -1
    draft[1, 2] = V
    pad = np.zeros(B, np.int32)
    got = _run_gpu(sd, tl, dl, draft, pad, ua, us, T, k + 1)
    check_against_oracle(tl, dl, "bf16", draft, pad, ua, us, T, k + 1, got)
    assert got["n_acc"][0] == 0 and got["n_acc"][1] <= 2
    t = tl.float().numpy()
    for i in range(B):
        assert np.isfinite(t[i, got["n_acc"][i], got["bonus"][i]]), "a masked token was drawn"


def test_verify_sample_flags_bad_uniforms(sd):
    """Uniforms outside [0, 1) are clamped and flagged."""
    rng = np.random.default_rng(12)
    B, k, V, T = 4, 2, 100, 1.0
    tl, dl, draft, ua, us = _make(rng, B, k, V, "f32", T)
    ua[0, 0] = 1.5
    us[1] = -0.25
    got = _run_gpu(sd, tl, dl, draft, np.zeros(B, np.int32), ua, us, T, k + 1)
    assert got["status"] == sd.DEV_BAD_UNIFORM


def test_verify_sample_then_realign(sd):
    """The outputs feed the realignment entry points unchanged: a sampled step
    followed by the out-of-place realign equals the oracle's realignment for
    the GPU's accepted counts."""
    from paper_2510_22876_amd import workloads as wl
    rng = np.random.default_rng(13)
    w = wl.WORKLOADS["tiny"]
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    tl, dl, draft, ua, us = _make(rng, w.B, w.k, w.V, "f32", 0.9)
    got = _run_gpu(sd, tl, dl, draft, pad_in, ua, us, 0.9, W_in)
    src = wl.make_kv(w, pad_in, W_in, cap, device="cuda")
    dst = torch.zeros_like(src)
    sd.specdec_realign_kv(src, dst, w.k, W_in, torch.as_tensor(pad_in, device="cuda"),
                          torch.as_tensor(got["n_acc"], device="cuda"),
                          torch.tensor([got["w_new"]], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    from tests.gpu_util import bits
    exp = oracle.realign_kv(bits(src), w.k, W_in, pad_in, got["n_acc"], got["w_new"])
    W = got["w_new"]
    assert np.array_equal(bits(dst)[..., :W, :], exp[..., :W, :])


@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_step_sample_equals_split_calls(sd, variant):
    """specdec_step_sample (one call) equals specdec_verify_sample followed by
    the realignment, position-id / mask and token-row entry points, bit for
    bit, on a vicuna7b-shaped batch with fewer layers."""
    from paper_2510_22876_amd import workloads as wl
    from tests.gpu_util import bits
    w = wl.WORKLOADS["vicuna7b"].scaled(L=2, H=4)
    rng = np.random.default_rng(14)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    tl, dl, draft, ua, us = _make(rng, w.B, w.k, w.V, "bf16", 0.8)
    dev = "cuda"
    T = 0.8
    src = wl.make_kv(w, pad_in, W_in, cap, device=dev)
    s_rows = wl.make_token_rows(w, pad_in, W_in, cap + 2, 0, -2, device=dev)
    outs = []
    for fused in (True, False):
        kv = src.clone()
        dst = torch.zeros_like(kv) if variant == "oop" else kv
        srow = s_rows.clone()
        s_out = torch.zeros((w.B, W_in + 1), dtype=torch.int32, device=dev) if variant == "oop" else srow
        i32 = dict(dtype=torch.int32, device=dev)
        o = dict(tokens=torch.zeros((w.B, w.k + 1), **i32), n_acc=torch.zeros(w.B, **i32), bonus=torch.zeros(w.B, **i32),
                 pad_out=torch.zeros(w.B, **i32), w_new=torch.zeros(1, **i32))
        pos = torch.zeros((w.B, W_in + w.k + 1), dtype=torch.int64, device=dev)
        mask = torch.zeros((w.B, W_in + w.k + 1), dtype=torch.uint8, device=dev)
        ws = sd.alloc_sample_workspace(w.B, w.k, w.V, dev)
        st = torch.zeros(1, **i32)
        args = (tl.to(dev), dl.to(dev), torch.as_tensor(draft, device=dev), torch.as_tensor(pad_in, device=dev),
                torch.as_tensor(ua, device=dev), torch.as_tensor(us, device=dev), T, W_in)
        if fused:
            wn = sd.specdec_step_sample(*args, kv, dst, o["tokens"], o["n_acc"], o["bonus"], o["pad_out"], o["w_new"],
                                        pos, mask, ws, st, sync_w_new=True, s_in=srow, s_out=s_out, pad_id=-2)
        else:
            sd.specdec_verify_sample(*args, o["tokens"], o["n_acc"], o["bonus"], o["pad_out"], o["w_new"], ws, st)
            sd.specdec_realign_kv(kv, dst, w.k, W_in, args[3], o["n_acc"], o["w_new"], st)
            sd.specdec_build_posmask(o["pad_out"], o["w_new"], w.k, pos, mask, st)
            sd.specdec_realign_tokens(srow, s_out, o["tokens"], args[3], o["n_acc"], o["w_new"], W_in, -2, st)
            wn = int(o["w_new"].cpu()[0])
        torch.cuda.synchronize()
        assert int(st.cpu()[0]) == 0
        W = wn
        outs.append((W, {n: t.cpu().numpy() for n, t in o.items()}, bits(dst)[..., :W, :],
                     pos.cpu().numpy()[:, :W + w.k + 1], mask.cpu().numpy()[:, :W + w.k + 1],
                     s_out.cpu().numpy()[:, :W + 1]))
    a, b = outs
    assert a[0] == b[0]
    for name in a[1]:
        assert np.array_equal(a[1][name], b[1][name]), name
    for x, y in zip(a[2:], b[2:]):
        assert np.array_equal(x, y)
