"""GPU parity: the HIP path, called through the C ABI, against the oracle.

Small shapes (several workgroup chunks and a ragged tail, every workload
family, both variants, both entry-point routes) are compared element by
element.  Edge cases: one row, uniform acceptance, all-reject / all-accept,
k = 0, empty old content, ragged vocabularies, V = 1, D = 8 / 256, a large
batch, the largest k, planted ties across workgroup boundaries, NaN / -0.0
rows, an unaligned logits pointer, an empty batch, workspace reuse, and device
values out of range (flagged, rows left untouched).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests import checker
from tests.gpu_util import (SENT_KV, alloc_outputs, bits, check_kv_full_vs_oracle, check_posmask_vs_oracle,
                            check_relocation_on_device, check_tokens_vs_oracle, check_verify_vs_oracle, i16, run_gpu,
                            say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec  # noqa: F401  (raises if the library is not built)
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _full_check(r):
    v = check_verify_vs_oracle(r)
    check_kv_full_vs_oracle(r, v)
    check_posmask_vs_oracle(r, v)
    check_relocation_on_device(r, r.out["pad_out"], r.out["n_acc"], r.out["w_new"])
    check_tokens_vs_oracle(r, v)
    if r.variant == "oop":
        # out of place: columns [w_new, cap) of the destination are untouched
        tail = i16(r.dst[..., r.out["w_new"]:, :])
        assert bool((tail == SENT_KV).all()), "destination written beyond w_new"
    return v


def _small(name, **kw):
    return wl.WORKLOADS[name].scaled(**kw)


SMALL = {
    "tiny": wl.WORKLOADS["tiny"],
    "vicuna7b_small": _small("vicuna7b", L=2, H=4, prompt=("uniform", 128, 1024)),
    "gqa8b_small": _small("gqa8b", L=2, H=2, prompt=("loguniform", 64, 4096)),
    "stress_small": _small("stress", B=16, L=1, H=2, prompt=("uniform", 512, 8192)),
    "f16_logits": _small("vicuna7b", logit_dtype="f16", V=32003, L=1, H=2, D=64, prompt=("uniform", 3, 300)),
}


@pytest.mark.parametrize("variant", ["oop", "inplace"])
@pytest.mark.parametrize("api", ["step", "split"])
@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_workloads(name, api, variant):
    # the token row rides along: out of place with the out-of-place cache, in
    # place with the in-place one
    for seed in (0, 1):
        _full_check(run_gpu(SMALL[name], seed=seed, variant=variant, api=api, tokens=variant))


@pytest.mark.parametrize("tok", ["oop", "inplace"])
@pytest.mark.parametrize("variant", ["oop", "inplace"])
@pytest.mark.parametrize("name", ["tiny", "empty_old_content", "k0", "max_k", "mixed_shift_signs", "large_batch"])
def test_token_rows(name, variant, tok):
    w = SMALL.get(name) or EDGE[name]
    for seed in (0, 2):
        _full_check(run_gpu(w, seed=seed, variant=variant, tokens=tok))


EDGE = {
    "one_row": _small("tiny", B=1, W_in=None, prompt=("fixed", 37)),
    "uniform_accept": _small("vicuna7b", L=1, H=2, D=16, V=500, accept=("fixed", 3), prompt=("uniform", 5, 90)),
    "all_reject": _small("vicuna7b", L=1, H=2, D=16, V=500, accept=("fixed", 0), prompt=("uniform", 5, 90)),
    "all_accept": _small("vicuna7b", L=1, H=2, D=16, V=500, accept=("fixed", 5), prompt=("uniform", 5, 90)),
    "k0": _small("vicuna7b", k=0, L=1, H=2, D=16, V=777, prompt=("uniform", 5, 90)),
    "empty_old_content": _small("vicuna7b", B=3, L=1, H=2, D=16, V=300, prompt=("list", [0, 7, 0])),
    "ragged_vocab_bf16": _small("gqa8b", B=4, V=1001, L=1, H=1, D=8, prompt=("uniform", 1, 40)),
    "ragged_vocab_f32": _small("tiny", V=1001, W_in=None, prompt=("uniform", 1, 40)),
    "ragged_vocab_f16": _small("tiny", V=999, logit_dtype="f16", W_in=None),
    "vocab_one": _small("tiny", V=1, W_in=None),
    "d8": _small("vicuna7b", L=1, H=3, D=8, V=600),
    "d256": _small("vicuna7b", L=1, H=1, D=256, V=600),
    "large_batch": _small("gqa8b", B=2048, k=3, V=64, L=1, H=1, D=8, prompt=("uniform", 1, 60)),
    "max_k": _small("tiny", B=3, k=64, V=50, W_in=None, prompt=("uniform", 0, 20)),
    "ties_across_chunks": _small("stress", B=8, V=40000, L=1, H=1, D=8, tie_frac=0.5, prompt=("uniform", 1, 50)),
    "mixed_shift_signs": _small("tiny", B=6, W_in=80, prompt=("uniform", 3, 60)),
}


@pytest.mark.parametrize("variant", ["oop", "inplace"])
@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_cases(name, variant):
    for seed in (0, 3):
        _full_check(run_gpu(EDGE[name], seed=seed, variant=variant))


@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_draft_cache_realigned_with_the_target_offsets(variant):
    """Alg. 1 realigns every cache with one set of offsets: a draft model's
    cache of its own (L, H, D) shape, realigned by a second call with the
    target step's pad_in / n_acc / w_new, against the oracle element by
    element."""
    from paper_2510_22876_amd import specdec as sd
    w = SMALL["vicuna7b_small"]
    r = run_gpu(w, seed=5, variant="oop")
    v = check_verify_vs_oracle(r)
    wd = w.scaled(L=3, H=1, D=64)
    src = wl.make_kv(wd, r.pad_in, r.W_in, r.cap, 7, device="cuda")
    before = bits(src)
    dst = src if variant == "inplace" else torch.full_like(src.view(torch.int16), SENT_KV).view(torch.bfloat16)
    dev = lambda a: torch.as_tensor(np.asarray(a, np.int32), device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_realign_kv(src, dst, w.k, r.W_in, dev(r.pad_in), dev(r.out["n_acc"]), dev([r.out["w_new"]]), status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    W = v["w_new"]
    exp = oracle.realign_kv(before, w.k, r.W_in, r.pad_in, v["n_acc"], W)
    got = bits(dst)
    assert np.array_equal(got[..., :W, :], exp[..., :W, :])


@pytest.mark.parametrize("variant,items", [("oop", 64 * 600), ("inplace", 256 * 30)])
def test_realign_split_over_launches(monkeypatch, variant, items):
    """The realignment (with pos/mask and the token row) split over many
    launches when one launch may hold only `items` work-items: a few spans
    per launch, so the in-place kernel's XCD rotation maps workgroups of one
    launch onto spans of others; still every span is moved once."""
    monkeypatch.setenv("SPECDEC_MAX_LAUNCH_ITEMS", str(items))
    try:
        for seed in (0, 5):
            _full_check(run_gpu(SMALL["vicuna7b_small"], seed=seed, variant=variant, tokens=variant))
    finally:
        monkeypatch.delenv("SPECDEC_MAX_LAUNCH_ITEMS", raising=False)


def test_uniform_acceptance_in_place_touches_nothing():
    """Corollary B.4: every offset is zero, so the in-place step writes no KV byte."""
    w = EDGE["uniform_accept"].scaled(extra_cap=9)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    src = wl.make_kv(w, pad_in, W_in, cap, device="cuda")
    src[..., W_in:, :] = 3.0          # stale columns beyond the cache must survive too
    before = src.clone()
    r = run_gpu(w, variant="inplace", src=src, pad_in=pad_in, W_in=W_in)
    assert np.array_equal(r.out["pad_out"], pad_in)
    assert torch.equal(i16(src), i16(before))


def test_special_logit_values():
    """NaN (first NaN wins), -0.0 vs +0.0, -inf rows, ties at the first and last index."""
    w = _small("tiny", B=4, k=2, V=37, W_in=None, prompt=("uniform", 2, 9))
    for dt in ("f32", "bf16", "f16"):
        x = torch.randn((w.B, w.k + 1, w.V)) * 0.5
        x[0, 0, 5] = float("nan"); x[0, 0, 30] = float("nan"); x[0, 0, 7] = 100.0
        x[0, 1] = -0.0; x[0, 1, 3] = 0.0
        x[0, 2] = float("-inf")
        x[1, 0, 0] = 50.0; x[1, 0, 36] = 50.0
        x[1, 1, 36] = 60.0
        x[1, 2] = 1.0
        x[2, :, 10] = float("inf"); x[2, :, 20] = float("inf")
        x[3, 0, :] = float("nan")
        logits = x.to(wl.TORCH_DT[dt]).cuda()
        ww = w.scaled(logit_dtype=dt)
        draft = torch.randint(0, w.V, (w.B, w.k), dtype=torch.int32)
        draft[1, 0] = 0
        r = run_gpu(ww, logits=logits, draft=draft.cuda())
        _full_check(r)
        assert r.out["tokens"][0, 0] == 5 and r.out["tokens"][1, 0] == 0 and r.out["tokens"][2, 0] == 10


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_nan_bit_patterns_16bit(dt):
    """16-bit NaNs of either sign and any payload rank above every number and
    the first one wins, inside 16-byte vectors and in unaligned heads / tails
    (rows of 1001 logits); a row whose only NaN is negative, and a row of
    -inf with one negative NaN."""
    V = 1001
    w = _small("tiny", B=6, k=2, V=V, W_in=None, prompt=("uniform", 2, 9)).scaled(logit_dtype=dt)
    neg = [0xFF81, 0xFFC0, 0xFFFF] if dt == "bf16" else [0xFC01, 0xFE00, 0xFFFF]
    pos = [0x7F81, 0x7FC0, 0x7FFF] if dt == "bf16" else [0x7C01, 0x7E00, 0x7FFF]
    x = (torch.randn((w.B, w.k + 1, V)) * 0.5).to(wl.TORCH_DT[dt]).view(torch.int16)
    def put(i, r, j, bits):
        x[i, r, j] = bits - 65536 if bits >= 32768 else bits
    put(0, 0, 500, neg[0]); put(0, 0, 700, pos[1])          # negative first: index 500
    put(0, 1, 3, neg[1])                                     # only NaN, in a row's head
    put(0, 2, V - 1, neg[2]); put(0, 2, 998, pos[0])         # the positive one comes first
    for j, b in zip((100, 101, 102), neg):                  # a run of payloads in one vector
        put(1, 0, j, b)
    x[1, 1] = torch.tensor(0xFF80 if dt == "bf16" else 0xFC00, dtype=torch.int32).to(torch.int16)  # -inf row
    put(1, 1, 640, neg[0])
    put(2, 0, 0, neg[2])                                     # at index 0
    logits = x.view(wl.TORCH_DT[dt]).cuda()
    draft = torch.randint(0, V, (w.B, w.k), dtype=torch.int32)
    r = run_gpu(w, logits=logits, draft=draft.cuda())
    _full_check(r)
    t = r.out["tokens"]
    assert (t[0, 0], t[0, 1], t[0, 2], t[1, 0], t[1, 1], t[2, 0]) == (500, 3, 998, 100, 640, 0)


def test_unaligned_logits_pointer():
    w = _small("gqa8b", B=3, V=997, L=1, H=1, D=8, prompt=("uniform", 1, 30))
    logits, draft, *_ = wl.logits_and_drafts(w, 0, 0, device="cuda")
    flat = torch.empty(logits.numel() + 1, dtype=logits.dtype, device="cuda")
    shifted = flat[1:].view_as(logits)
    shifted.copy_(logits)
    assert shifted.data_ptr() % 16 != 0
    _full_check(run_gpu(w, logits=shifted, draft=draft))


def test_empty_batch_is_a_noop():
    from paper_2510_22876_amd import specdec as sd
    o = alloc_outputs(1, 2, 50, 10)
    e = torch.empty((0, 3, 50), dtype=torch.bfloat16, device="cuda")
    d = torch.empty((0, 2), dtype=torch.int32, device="cuda")
    z = torch.empty(0, dtype=torch.int32, device="cuda")
    t = torch.empty((0, 3), dtype=torch.int32, device="cuda")
    sd.specdec_verify_greedy(e, d, z, 8, t, z, z, z, o.w_new, o.workspace)
    torch.cuda.synchronize()
    assert int(o.w_new.cpu()[0]) == -99


def test_workspace_reused_across_calls():
    """Consecutive calls on one workspace (filled with garbage first) with
    different inputs all agree with the oracle: the workspace needs no
    initialisation."""
    from paper_2510_22876_amd import specdec as sd
    w = SMALL["vicuna7b_small"]
    o = alloc_outputs(w.B, w.k, w.V, 2000)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    pad_t = torch.as_tensor(pad_in, device="cuda")
    o.workspace.fill_(0x5A5A5A5A5A5A5A5A)
    for seed in range(5):
        logits, draft, *_ = wl.logits_and_drafts(w, seed, seed, device="cuda")
        say(f"workspace reuse call {seed}")
        sd.specdec_verify_greedy(logits, draft, pad_t, W_in, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                                 o.workspace, o.dev_status)
        torch.cuda.synchronize()
        v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), pad_in, W_in)
        assert np.array_equal(o.tokens.cpu().numpy(), v["tokens"])
        assert np.array_equal(o.n_acc.cpu().numpy(), v["n_acc"])
        assert int(o.w_new.cpu()[0]) == v["w_new"]


def test_out_of_range_device_values_are_flagged():
    """pad_in / n_acc out of range (forced from the host): the kernels flag them
    in dev_status and leave those rows untouched; the other rows still follow
    the oracle for the width computed over the valid rows."""
    from paper_2510_22876_amd import specdec as sd
    w = _small("vicuna7b", B=4, L=1, H=2, D=16, V=300, prompt=("uniform", 5, 40))
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    W0 = W_in - (w.k + 1)
    bad = pad_in.copy()
    bad[1] = -1
    bad[2] = W0 + 5
    logits, draft, *_ = wl.logits_and_drafts(w, 0, 0, device="cuda")
    src = wl.make_kv(w, pad_in, W_in, cap, device="cuda")
    dst = torch.full_like(i16(src), SENT_KV).view(torch.bfloat16)
    o = alloc_outputs(w.B, w.k, w.V, W_in + w.k + 1)
    sd.specdec_step(logits, draft, torch.as_tensor(bad, device="cuda"), W_in, src, dst, o.tokens, o.n_acc,
                    o.bonus, o.pad_out, o.w_new, o.pos, o.mask, o.workspace, o.dev_status)
    torch.cuda.synchronize()
    st = int(o.dev_status.cpu()[0])
    assert st & sd.DEV_BAD_PAD_IN and st & sd.DEV_BAD_PAD_OUT
    pad_out = o.pad_out.cpu().numpy()
    assert pad_out[1] == -1 and pad_out[2] == -1
    good = [0, 3]
    v = oracle.verify(logits.cpu()[good], w.logit_dtype, draft.cpu().numpy()[good], pad_in[good], W_in)
    assert int(o.w_new.cpu()[0]) == v["w_new"]
    got = bits(dst)
    exp = oracle.realign_kv(bits(src)[:, :, good], w.k, W_in, pad_in[good], v["n_acc"], v["w_new"])
    assert np.array_equal(got[:, :, good, :, : v["w_new"]], exp[..., : v["w_new"], :])
    assert np.all(got[:, :, [1, 2]] == SENT_KV), "rows with invalid values must be left untouched"
    # an out-of-range accepted count handed to the realign entry point alone
    o.dev_status.zero_()
    n_acc = o.n_acc.clone()
    n_acc[0] = w.k + 3
    dst2 = torch.full_like(i16(src), SENT_KV).view(torch.bfloat16)
    sd.specdec_realign_kv(src, dst2, w.k, W_in, torch.as_tensor(pad_in, device="cuda"), n_acc, o.w_new,
                          o.dev_status)
    torch.cuda.synchronize()
    assert int(o.dev_status.cpu()[0]) & sd.DEV_BAD_ACCEPT
    assert bool((i16(dst2[:, :, 0]) == SENT_KV).all())
