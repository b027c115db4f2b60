"""specdec_step_noalloc (the fused step on the library's own scratch, for
callers that cannot allocate) against specdec_step with a caller workspace,
through the C ABI: every output bit for bit, on consecutive calls that share
the library scratch, each later one smaller.  The first two cases have
logit rows longer than 16 KB (verification in the scan and merge launches,
partial maxima in the scratch); the others verify in one launch (one
workgroup per row, completion counted in the scratch), including planted
ties, f16 logits, k = 0 and a row whose pad_in is out of range.  Both calls of a pair see
identical input bytes and identically pre-filled output buffers, and the
verification outputs are also checked against the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests.gpu_util import PAD_ID, SENT_KV, SENT_MASK, SENT_POS, SENT_TOK, alloc_outputs, say

pytestmark = pytest.mark.gpu

SHAPES = [
    # (name, workload overrides): each later case is smaller than the one before it
    ("vicuna7b", dict(B=4, V=70000, L=2, H=2, D=128, prompt=("uniform", 64, 300))),     # rows of 140 KB
    ("vicuna7b", dict(B=8, V=32000, L=2, H=4, D=64, prompt=("uniform", 32, 200))),
    ("stress", dict(B=6, V=4099, L=1, H=2, D=16, prompt=("uniform", 3, 50), tie_frac=0.25)),
    ("gqa8b", dict(B=5, V=3001, L=1, H=2, D=64, prompt=("loguniform", 4, 120))),
    ("tiny", dict(logit_dtype="f16", logit_std=3.0, V=777)),
    ("tiny", dict(k=0, B=1, V=500)),
]


def _workload(name, over):
    return wl.WORKLOADS[name].scaled(**over) if over else wl.WORKLOADS[name]


def _inputs(w, seed, bad_row=None):
    n, W_in, pad_in, cap = wl.initial_geometry(w, seed)
    logits, draft, *_ = wl.logits_and_drafts(w, seed, 0, device="cuda")
    src = wl.make_kv(w, pad_in, W_in, cap, seed, device="cuda")
    s_rows = wl.make_token_rows(w, pad_in, W_in, cap + 2, seed, PAD_ID, device="cuda")
    if bad_row is not None:
        pad_in = pad_in.copy()
        pad_in[bad_row] = W_in - (w.k + 1) + 1          # outside [0, L]: flagged, the row left out
    return W_in, cap, pad_in, logits, draft, src, s_rows


def _one(sd, w, W_in, cap, pad_in, logits, draft, src, s_rows, variant, noalloc):
    pm_cap = W_in + w.k + 1 + 3
    o = alloc_outputs(w.B, w.k, w.V, pm_cap)
    pad_t = torch.as_tensor(np.asarray(pad_in, np.int32), device="cuda")
    if variant == "oop":
        s = src
        d = torch.full(src.shape, SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        s_in = s_rows
        s_out = torch.full((w.B, W_in + 1 + 5), SENT_TOK, dtype=torch.int32, device="cuda")
    else:
        s = d = src.clone()
        s_in = s_out = s_rows.clone()
    args = (logits, draft, pad_t, W_in, s, d, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new, o.pos, o.mask)
    if noalloc:
        wn = sd.specdec_step_noalloc(*args, o.dev_status, sync_w_new=True, s_in=s_in, s_out=s_out, pad_id=PAD_ID)
    else:
        o.workspace.fill_(0x3C3C3C3C3C3C3C3C)
        wn = sd.specdec_step(*args, o.workspace, o.dev_status, sync_w_new=True, s_in=s_in, s_out=s_out, pad_id=PAD_ID)
    torch.cuda.synchronize()
    out = {name: getattr(o, name).cpu().numpy() for name in ("tokens", "n_acc", "bonus", "pad_out", "w_new", "pos",
                                                             "mask", "dev_status")}
    out["kv"] = d.view(torch.int16).cpu().numpy()
    out["s_out"] = s_out.cpu().numpy()
    out["w_host"] = wn
    return out


def _against_oracle(w, W_in, pad_in, logits, draft, got):
    v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), pad_in, W_in)
    assert np.array_equal(got["tokens"], v["tokens"]) and np.array_equal(got["n_acc"], v["n_acc"])
    assert np.array_equal(got["bonus"], v["bonus"])
    assert int(got["w_new"][0]) == v["w_new"]


@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_noalloc_step_equals_step(variant):
    """The reference outputs first (caller workspace filled with garbage),
    then the no-alloc calls back to back from the largest case to the
    smallest, all on the same library scratch."""
    from paper_2510_22876_amd import specdec as sd
    cases = []
    for i, (name, over) in enumerate(SHAPES):
        w = _workload(name, over)
        cases.append((name, w, _inputs(w, seed=i)))
    refs = []
    for name, w, inp in cases:
        say(f"step (workspace): {name} B={w.B} k={w.k} V={w.V} {w.logit_dtype} L={w.L} H={w.H} D={w.D} {variant}")
        refs.append(_one(sd, w, *inp, variant, noalloc=False))
    for (name, w, inp), ref in zip(cases, refs):
        say(f"step_noalloc: {name} B={w.B} k={w.k} V={w.V} {w.logit_dtype} L={w.L} H={w.H} D={w.D} {variant}")
        got = _one(sd, w, *inp, variant, noalloc=True)
        assert int(ref["dev_status"][0]) == 0 and int(got["dev_status"][0]) == 0
        for key in ref:
            assert np.array_equal(np.asarray(ref[key]), np.asarray(got[key])), (name, variant, key)
        assert got["w_host"] == int(ref["w_new"][0])
        W_in, cap, pad_in, logits, draft, *_ = inp
        _against_oracle(w, W_in, pad_in, logits, draft, got)


def test_noalloc_consecutive_one_launch_verifications():
    """Ten one-launch verifications in a row of changing batch size, each
    equal to specdec_step: the realignment clears the completion counts that
    the next call's verification starts from."""
    from paper_2510_22876_amd import specdec as sd
    for t, B in enumerate([8, 3, 8, 1, 5, 2, 8, 7, 1, 4]):
        w = _workload("vicuna7b", dict(B=B, V=5000 + 97 * t, L=1, H=2, D=16, prompt=("uniform", 8, 60)))
        say(f"consecutive one-launch call {t}: B={B} V={w.V}")
        inp = _inputs(w, seed=40 + t)
        ref = _one(sd, w, *inp, "oop", noalloc=False)
        got = _one(sd, w, *inp, "oop", noalloc=True)
        for key in ref:
            assert np.array_equal(np.asarray(ref[key]), np.asarray(got[key])), (t, key)


def test_noalloc_bad_pad_in_flagged_like_step():
    """A row whose pad_in lies outside [0, L] is flagged and left out of the
    width by the one-launch verification exactly as by specdec_step."""
    from paper_2510_22876_amd import specdec as sd
    w = _workload("vicuna7b", dict(B=4, V=3001, L=1, H=2, D=16, prompt=("uniform", 8, 60)))
    say("bad pad_in: B=4 V=3001, row 1 out of range")
    inp = _inputs(w, seed=7, bad_row=1)
    ref = _one(sd, w, *inp, "oop", noalloc=False)
    got = _one(sd, w, *inp, "oop", noalloc=True)
    assert int(ref["dev_status"][0]) & sd.DEV_BAD_PAD_IN
    for key in ref:
        assert np.array_equal(np.asarray(ref[key]), np.asarray(got[key])), key
    assert int(got["pad_out"][1]) == -1


def test_noalloc_rejects_beyond_its_scratch():
    """A step whose verification needs more than the library's scratch is
    refused with SPECDEC_ERR_WORKSPACE before anything is enqueued."""
    from paper_2510_22876_amd import specdec as sd
    B, k, V = 16384, 7, 128256
    assert sd.workspace_bytes(B, k, V) > 4194304
    logits = torch.empty((B, k + 1, V), dtype=torch.bfloat16, device="cuda")   # 34 GB, never read
    draft = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    pad_t = torch.zeros(B, dtype=torch.int32, device="cuda")
    kv = torch.zeros((1, 2, B, 1, 16, 8), dtype=torch.bfloat16, device="cuda")
    dst = torch.zeros_like(kv)
    o = alloc_outputs(B, k, 16, 16 + k + 1)   # small V: only the output buffers are used
    with pytest.raises(sd.SpecdecError) as e:
        sd.specdec_step_noalloc(logits, draft, pad_t, 16, kv, dst, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                                o.pos, o.mask, o.dev_status)
    assert e.value.code == sd.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert int(o.w_new.cpu()[0]) == -99        # nothing ran


@pytest.mark.parametrize("V", [5000, 32000], ids=["one_launch_verify", "two_launch_verify"])
def test_noalloc_step_replayed_from_a_graph(V):
    """The caller this entry point is for: the step captured once in a HIP
    graph and replayed on new inputs (eager copies and synchronisations in
    between), each replay equal to an eager specdec_step with a caller
    workspace, bit for bit.  Replays of the one-launch verification rely on
    the realignment launch clearing the completion counts for the next
    replay."""
    from paper_2510_22876_amd import specdec as sd
    sd.timing_enable(False)     # kernel timers record events: none inside the capture
    w = _workload("vicuna7b", dict(B=6, V=V, L=2, H=2, D=64, prompt=("uniform", 16, 120)))
    n, W_in, pad_in, cap = wl.initial_geometry(w, 3)
    src0 = wl.make_kv(w, pad_in, W_in, cap, 3, device="cuda")
    inputs = [wl.logits_and_drafts(w, 3, t, device="cuda")[:2] for t in range(4)]
    pad_t = torch.as_tensor(np.asarray(pad_in, np.int32), device="cuda")
    lg = inputs[0][0].clone()
    dr = inputs[0][1].clone()
    src = src0.clone()
    dst = torch.empty_like(src0)
    o = alloc_outputs(w.B, w.k, w.V, W_in + w.k + 1)

    def step():
        sd.specdec_step_noalloc(lg, dr, pad_t, W_in, src, dst, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                                o.pos, o.mask, o.dev_status)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                  # warm-up (and the scratch's first use) outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    seen = set()
    for t in (1, 2, 3, 1, 2):
        say(f"noalloc graph replay V={V} inputs={t}")
        e = alloc_outputs(w.B, w.k, w.V, W_in + w.k + 1)
        e_dst = torch.empty_like(src0)
        sd.specdec_step(inputs[t][0], inputs[t][1], pad_t, W_in, src0, e_dst, e.tokens, e.n_acc, e.bonus, e.pad_out,
                        e.w_new, e.pos, e.mask, e.workspace, e.dev_status)
        torch.cuda.synchronize()
        lg.copy_(inputs[t][0])
        dr.copy_(inputs[t][1])
        for x in (o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new):
            x.fill_(-77)
        o.pos.fill_(SENT_POS)       # columns past w_new + k + 1 are left as they are:
        o.mask.fill_(SENT_MASK)     # the same sentinels as the eager outputs
        dst.view(torch.int16).fill_(0x7FC1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        W = int(e.w_new.cpu()[0])
        assert int(o.dev_status.cpu()[0]) == 0 and int(e.dev_status.cpu()[0]) == 0
        for name in ("tokens", "n_acc", "bonus", "pad_out", "w_new", "pos", "mask"):
            assert np.array_equal(getattr(o, name).cpu().numpy(), getattr(e, name).cpu().numpy()), (t, name)
        assert np.array_equal(dst[..., :W, :].view(torch.int16).cpu().numpy(),
                              e_dst[..., :W, :].view(torch.int16).cpu().numpy()), (t, "kv")
        seen.add(tuple(o.n_acc.cpu().tolist()))
    assert len(seen) > 1, "the replays should see different acceptance patterns"
