"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (the fused step).

The oracle computes verification over every logit row, position ids / mask
over every row, and the KV relocation of sampled spans (every row, the first
and last span, random extras; K and V each).  The whole cache is checked with
torch on the device against the relocation property (pads +0.0, content equal
to the kept source columns) and, for the in-place variant, against the
out-of-place result.  The chained workload runs 16 in-place steps on tagged
KV and checks the cache clause of I2 (Theorem B.1) after every 4th step and
the last.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_22876_amd import workloads as wl
from tests import checker
from tests.gpu_util import (PAD_ID, alloc_outputs, check_posmask_vs_oracle, check_relocation_on_device,
                            check_spans_vs_oracle, check_tokens_vs_oracle, check_verify_vs_oracle, host_spans, i16,
                            run_gpu, sample_spans, say)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec  # noqa: F401
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["vicuna7b", "gqa8b", "stress"])
def test_full_size(name):
    w = wl.WORKLOADS[name]
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    spans = sample_spans(w)
    logits, draft, *_ = wl.logits_and_drafts(w, 0, 0, device="cuda")
    src = wl.make_kv(w, pad_in, W_in, cap, device="cuda")
    src_spans = host_spans(src, spans, W_in)
    r = run_gpu(w, variant="oop", logits=logits, draft=draft, src=src, pad_in=pad_in, W_in=W_in, tokens="oop")
    v = check_verify_vs_oracle(r)
    check_posmask_vs_oracle(r, v)
    check_tokens_vs_oracle(r, v)
    check_spans_vs_oracle(w, spans, src_spans, host_spans(r.dst, spans, W_in), pad_in, v, W_in)
    check_relocation_on_device(r, v["pad_out"], v["n_acc"], v["w_new"])
    say(f"{name}: out-of-place checked, w_new={v['w_new']}, n_acc={v['n_acc'].tolist()[:16]}")
    oop = r.dst
    W = v["w_new"]
    # in place on the same input, then against the out-of-place result
    r2 = run_gpu(w, variant="inplace", logits=logits, draft=draft, src=src, pad_in=pad_in, W_in=W_in,
                 keep_src=False)
    del r
    assert r2.out["w_new"] == W
    assert np.array_equal(r2.out["n_acc"], v["n_acc"])
    check_spans_vs_oracle(w, spans, src_spans, host_spans(src, spans, W_in), pad_in, v, W_in)
    for l in range(w.L):
        assert torch.equal(i16(src[l, :, :, :, :W, :]), i16(oop[l, :, :, :, :W, :])), f"in place != out of place, layer {l}"
    say(f"{name}: in-place checked")


def test_chained_in_place_tagged():
    w = wl.WORKLOADS["vicuna7b_chained"]
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    kv = wl.make_kv(w, pad_in, W_in, cap, device="cuda", tagged=True)
    prod = [np.zeros(int(n[i]), np.int64) for i in range(w.B)]
    pad = pad_in.copy()
    W0 = W_in - (w.k + 1)
    spans = sample_spans(w, n_extra=4)
    s_rows = wl.make_token_rows(w, pad_in, W_in, cap + 2, 0, PAD_ID, device="cuda")
    model = [list(s_rows[i, pad_in[i]:W_in - w.k].cpu().numpy()) for i in range(w.B)]
    for step in range(w.steps):
        if step > 0:
            wl.write_window(kv, w, W0, pad, seed=0, step=step, tagged=True)
        Wi = W0 + w.k + 1
        assert Wi <= cap
        logits, draft, *_ = wl.logits_and_drafts(w, 0, step, device="cuda")
        src_spans = host_spans(kv, spans, Wi)
        say(f"chained step {step}: W_in={Wi}")
        r = run_gpu(w, variant="inplace", logits=logits, draft=draft, src=kv, pad_in=pad, W_in=Wi,
                    tokens="inplace", s_rows=s_rows)
        v = check_verify_vs_oracle(r)
        check_posmask_vs_oracle(r, v)
        check_tokens_vs_oracle(r, v)
        d = draft.cpu().numpy()
        for i in range(w.B):   # Alg. 1's append, replayed per sequence
            model[i] += list(d[i, : v["n_acc"][i]]) + [v["bonus"][i]]
            assert list(r.extra["s_out"][i, v["pad_out"][i]: v["w_new"] + 1]) == model[i]
        check_spans_vs_oracle(w, spans, src_spans, host_spans(kv, spans, Wi), pad, v, Wi)
        check_relocation_on_device(r, v["pad_out"], v["n_acc"], v["w_new"])
        prod = checker.advance_prod_steps(prod, W0 - pad, v["n_acc"], step)
        if step % 4 == 3 or step == w.steps - 1:
            checker.check_tagged_kv_device(kv, v["pad_out"], v["w_new"], prod)
            say(f"chained step {step}: tags checked")
        del r
        pad, W0 = v["pad_out"].copy(), v["w_new"]


@pytest.mark.parametrize("batch_kind", ["ragged", "same"])
def test_exspec_full_size(batch_kind):
    """EXSpec's step at the vicuna7b shape in the benchmark's configuration
    (pool of 32 sequences, the first 8 gathered, verified, written back in
    append mode): paddings, token rows and pos/mask against the oracle in
    full; sampled (layer, row, head) spans of the batch and of the pool after
    write-back against the oracle; every row of the batch and every slot with
    torch on the device against the gather / write-back definitions."""
    from paper_2510_22876_amd import specdec as sd
    w = wl.WORKLOADS["vicuna7b"]
    B, k = w.B, w.k
    N = 4 * B
    lens = wl.pool_lengths(w, N, 0)
    if batch_kind == "same":
        lens[:B] = lens[0]
    slots = np.arange(B, dtype=np.int32)
    Lb = int(lens[:B].max())
    cap = int(lens.max()) + 2 * (k + 1)
    say(f"exspec full size {batch_kind}: N={N} Lb={Lb} cap={cap}")
    pool, pool_tok = wl.make_pool(w, lens, cap, cap + 2, 0, device="cuda")
    spans = sample_spans(w)
    pool_before = {s: i16(pool[s[0], :, s[1], s[2], :cap, :]).cpu().numpy().view(np.uint16) for s in spans}
    tok_before = pool_tok.cpu().numpy()
    bcap = Lb + k + 1
    batch = torch.empty((w.L, 2, B, w.H, bcap, w.D), dtype=torch.bfloat16, device="cuda")
    btok = torch.empty((B, bcap + 1), dtype=torch.int32, device="cuda")
    pads = torch.empty(B, dtype=torch.int32, device="cuda")
    pos = torch.empty((B, bcap), dtype=torch.int64, device="cuda")
    mask = torch.empty((B, bcap), dtype=torch.uint8, device="cuda")
    lens_d = torch.as_tensor(lens, device="cuda")
    slots_d = torch.as_tensor(slots, device="cuda")
    logits, draft, *_ = wl.logits_and_drafts(w, 0, 0, device="cuda")
    o = alloc_outputs(B, k, w.V, bcap)
    sd.specdec_gather_batch(pool, pool_tok, lens_d, slots_d, Lb, batch, pads, batch_tok=btok, pos=pos, mask=mask,
                            k=k, pad_id=PAD_ID, dev_status=o.dev_status)
    wl.write_window(batch, w, Lb, Lb - lens[:B], seed=0, step=1)
    sd.specdec_verify_greedy(logits, draft, pads, Lb + k + 1, o.tokens, o.n_acc, o.bonus, o.pad_out, o.w_new,
                             o.workspace, o.dev_status)
    batch_spans = host_spans(batch, spans, bcap)
    sd.specdec_scatter_accepted(batch, pads, o.tokens, o.n_acc, slots_d, Lb, pool, pool_tok, lens_d,
                                batch_tok=btok, mode=sd.WRITEBACK_APPEND, dev_status=o.dev_status)
    torch.cuda.synchronize()
    assert int(o.dev_status.cpu()[0]) == 0
    pads_h = pads.cpu().numpy()
    assert np.array_equal(pads_h, Lb - lens[:B])
    if batch_kind == "same":
        assert not pads_h.any()
    n_acc = o.n_acc.cpu().numpy()
    v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), pads_h, Lb + k + 1)
    assert np.array_equal(n_acc, v["n_acc"]) and np.array_equal(o.tokens.cpu().numpy(), v["tokens"])
    # pos / mask and token rows in full
    epos, emask = oracle.posmask(pads_h, Lb, k, bcap)
    assert np.array_equal(pos.cpu().numpy(), epos) and np.array_equal(mask.cpu().numpy(), emask)
    exp_tok = tok_before.copy()
    exp_lens = lens.copy()
    # sampled spans: the gather against the oracle on the span, then the write-back
    for s in spans:
        l, i, h = s
        one = pool_before[(l, slots[i], h)] if (l, slots[i], h) in pool_before else \
            i16(pool[l, :, slots[i], h, :cap, :]).cpu().numpy().view(np.uint16)
        got = batch_spans[s]
        eb, _, _ = oracle.gather_batch(one.reshape(1, 2, 1, 1, cap, w.D), tok_before[slots[i]:slots[i] + 1],
                                       lens[slots[i]:slots[i] + 1], np.zeros(1, np.int32), Lb, bcap, bcap + 1, PAD_ID)
        assert np.array_equal(got[:, :Lb], eb.reshape(2, bcap, w.D)[:, :Lb]), f"gathered span {s} differs"
    # the whole batch and pool on the device: pads +0.0, content = the slot's entries, appended entries
    for i in range(B):
        p, n, a = int(pads_h[i]), int(lens[i]), int(n_acc[i]) + 1
        if p:
            assert bool((i16(batch[:, :, i, :, :p, :]) == 0).all()), f"row {i}: pads not +0.0"
        assert torch.equal(i16(batch[:, :, i, :, p:Lb, :]), i16(pool[:, :, slots[i], :, :n, :])), f"row {i} content"
        assert torch.equal(i16(pool[:, :, slots[i], :, n:n + a, :]), i16(batch[:, :, i, :, Lb:Lb + a, :])), \
            f"slot {slots[i]}: appended entries"
    eb_all, et_all, ep_all = oracle.gather_batch(np.zeros((1, 2, N, 1, cap, 8), np.uint16), tok_before, lens, slots,
                                                 Lb, bcap, bcap + 1, PAD_ID)
    oracle.scatter_accepted(eb_all, ep_all, v["tokens"], v["n_acc"], slots, Lb,
                            np.zeros((1, 2, N, 1, cap, 8), np.uint16), exp_tok, exp_lens, batch_tok=et_all)
    assert np.array_equal(lens_d.cpu().numpy(), exp_lens)
    assert np.array_equal(pool_tok.cpu().numpy(), exp_tok)
    got_btok = btok.cpu().numpy()
    for i in range(B):   # columns [0, Lb + 1 + a): the gathered row and the appended tokens
        end = Lb + 2 + int(n_acc[i])
        assert np.array_equal(got_btok[i, :end], et_all[i, :end]), f"batch token row {i}"
    say(f"exspec full size {batch_kind}: checked, n_acc={n_acc.tolist()}")
