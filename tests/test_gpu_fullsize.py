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
