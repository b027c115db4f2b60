"""specdec_step_noalloc (the fused step on the library's own scratch, for
callers that cannot allocate) against specdec_step with a caller workspace,
through the C ABI: every output bit for bit, on consecutive calls that share
the library scratch, the second with a smaller batch, vocabulary and cache.
Both calls of a pair see identical input bytes and identically pre-filled
output buffers."""
import numpy as np
import pytest
import torch

from paper_2510_22876_amd import workloads as wl
from tests.gpu_util import PAD_ID, SENT_KV, SENT_TOK, alloc_outputs, say

pytestmark = pytest.mark.gpu

SHAPES = [
    # (name, workload overrides): each later case is smaller than the one before it
    ("vicuna7b", dict(B=8, V=32000, L=2, H=4, D=128, prompt=("uniform", 64, 300))),
    ("gqa8b", dict(B=5, V=3001, L=1, H=2, D=64, prompt=("loguniform", 4, 120))),
    ("tiny", dict()),
]


def _inputs(w, seed):
    n, W_in, pad_in, cap = wl.initial_geometry(w, seed)
    logits, draft, *_ = wl.logits_and_drafts(w, seed, 0, device="cuda")
    src = wl.make_kv(w, pad_in, W_in, cap, seed, device="cuda")
    s_rows = wl.make_token_rows(w, pad_in, W_in, cap + 2, seed, PAD_ID, device="cuda")
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


@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_noalloc_step_equals_step(variant):
    """The reference outputs first (caller workspace filled with garbage),
    then the no-alloc calls back to back from the largest case to the
    smallest, all on the same library scratch."""
    from paper_2510_22876_amd import specdec as sd
    cases = []
    for i, (name, over) in enumerate(SHAPES):
        w = wl.WORKLOADS[name].scaled(**over) if over else wl.WORKLOADS[name]
        cases.append((name, w, _inputs(w, seed=i)))
    refs = []
    for name, w, inp in cases:
        say(f"step (workspace): {name} B={w.B} k={w.k} V={w.V} L={w.L} H={w.H} D={w.D} variant={variant}")
        refs.append(_one(sd, w, *inp, variant, noalloc=False))
    for (name, w, inp), ref in zip(cases, refs):
        say(f"step_noalloc: {name} B={w.B} k={w.k} V={w.V} L={w.L} H={w.H} D={w.D} variant={variant}")
        got = _one(sd, w, *inp, variant, noalloc=True)
        assert int(ref["dev_status"][0]) == 0 and int(got["dev_status"][0]) == 0
        for key in ref:
            assert np.array_equal(np.asarray(ref[key]), np.asarray(got[key])), (name, variant, key)
        assert got["w_host"] == int(ref["w_new"][0])


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
