"""The fused step captured in a HIP graph and replayed with new inputs.

torch.cuda.CUDAGraph records the library's launches on the capture stream
(the binding passes the current stream).  Nothing in the step allocates,
clears memory or synchronises when no host copy of the width is asked for,
so the whole step is capturable.  Each replay runs on new logits and drafts
copied into the captured input buffers, with eager work (copies, output
fills) and synchronisations between the replays, and must equal an eager call
on the same inputs bit for bit: tokens, counts, bonus, paddings, width,
positions, mask, token row and every cache byte up to the new width.
The step bound once (``specdec.bind_step``) and called on new contents of the
same buffers is held to the same bar.
"""
import numpy as np
import pytest
import torch

from paper_2510_22876_amd import workloads as wl
from tests.gpu_util import PAD_ID, bits, say

pytestmark = pytest.mark.gpu

W = wl.WORKLOADS["vicuna7b"].scaled(L=2, H=4, prompt=("uniform", 100, 700))


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec
    yield specdec
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _inputs(step, sample):
    if sample:
        lg, dlg, dr, ua, us = wl.sampled_inputs(W, 0, step, device="cuda")
        return dict(logits=lg, draft_logits=dlg, draft=dr, u_accept=ua, u_sample=us)
    lg, dr, *_ = wl.logits_and_drafts(W, 0, step, device="cuda")
    return dict(logits=lg, draft=dr)


class _Step:
    """Static buffers of one step and a call on them."""

    def __init__(self, sd, variant, sample, src0, pad_in, W_in, inp):
        self.sd, self.sample, self.W_in = sd, sample, W_in
        self.inp = {n: t.clone() for n, t in inp.items()}
        self.pad = torch.as_tensor(pad_in, device="cuda")
        self.src = src0.clone()
        self.dst = self.src if variant == "inplace" else torch.empty_like(src0)
        self.bufs = sd.StepBuffers(W.B, W.k, W.V, W_in + W.k + 1)
        if sample:
            self.bufs.workspace = sd.alloc_sample_workspace(W.B, W.k, W.V)
        self.s_in = wl.make_token_rows(W, pad_in, W_in, W_in + 2, 0, PAD_ID, device="cuda")
        self.s_out = self.s_in if variant == "inplace" else torch.empty_like(self.s_in)

    def load(self, inp, src0, s0):
        for n, t in inp.items():
            self.inp[n].copy_(t)
        self.src.copy_(src0)
        self.s_in.copy_(s0)
        for t in (self.bufs.tokens, self.bufs.n_acc, self.bufs.bonus, self.bufs.pad_out, self.bufs.w_new):
            t.fill_(-77)
        self.bufs.pos.fill_(-5)
        self.bufs.mask.fill_(9)
        if self.dst is not self.src:
            self.dst.view(torch.int16).fill_(0x7FC1)

    def __call__(self):
        b, i = self.bufs, self.inp
        if self.sample:
            self.sd.specdec_step_sample(i["logits"], i["draft_logits"], i["draft"], self.pad, i["u_accept"],
                                        i["u_sample"], 1.0, self.W_in, self.src, self.dst, b.tokens, b.n_acc,
                                        b.bonus, b.pad_out, b.w_new, b.pos, b.mask, b.workspace, b.dev_status,
                                        s_in=self.s_in, s_out=self.s_out, pad_id=PAD_ID)
        else:
            self.sd.specdec_step(i["logits"], i["draft"], self.pad, self.W_in, self.src, self.dst, b.tokens, b.n_acc,
                                 b.bonus, b.pad_out, b.w_new, b.pos, b.mask, b.workspace, b.dev_status,
                                 s_in=self.s_in, s_out=self.s_out, pad_id=PAD_ID)

    def result(self):
        b = self.bufs
        w = int(b.w_new.cpu()[0])
        return dict(tokens=b.tokens.cpu().numpy(), n_acc=b.n_acc.cpu().numpy(), bonus=b.bonus.cpu().numpy(),
                    pad_out=b.pad_out.cpu().numpy(), w_new=w, pos=b.pos.cpu().numpy(), mask=b.mask.cpu().numpy(),
                    status=int(b.dev_status.cpu()[0]), kv=bits(self.dst[..., :w, :]),
                    s_out=self.s_out.cpu().numpy()[:, :w + 1])


@pytest.mark.parametrize("sample", [False, True], ids=["greedy", "sample"])
@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_step_replayed_from_a_graph(sd, variant, sample):
    sd.timing_enable(False)            # kernel timers record events: none inside the capture
    n, W_in, pad_in, cap = wl.initial_geometry(W, 0)
    src0 = wl.make_kv(W, pad_in, W_in, cap, 0, device="cuda")
    s0 = wl.make_token_rows(W, pad_in, W_in, W_in + 2, 0, PAD_ID, device="cuda")
    inputs = [_inputs(t, sample) for t in range(5)]
    eager = _Step(sd, variant, sample, src0, pad_in, W_in, inputs[0])
    graphed = _Step(sd, variant, sample, src0, pad_in, W_in, inputs[0])
    # warm-up on a side stream, then capture
    graphed.load(inputs[0], src0, s0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        graphed()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed()
    torch.cuda.synchronize()
    accepted = set()
    for t in (1, 2, 3, 4, 1):
        say(f"graph replay variant={variant} sample={sample} inputs={t}")
        eager.load(inputs[t], src0, s0)
        eager()
        torch.cuda.synchronize()
        want = eager.result()
        graphed.load(inputs[t], src0, s0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = graphed.result()
        assert want["status"] == 0 and got["status"] == 0
        for name in want:
            assert np.array_equal(np.asarray(got[name]), np.asarray(want[name])), f"inputs {t}: {name} differs"
        accepted.add(tuple(got["n_acc"].tolist()))
    assert len(accepted) > 1, "the replays should see different acceptance patterns"


@pytest.mark.parametrize("noalloc", [False, True], ids=["workspace", "noalloc"])
@pytest.mark.parametrize("variant", ["oop", "inplace"])
def test_bound_step_equals_the_plain_call(sd, variant, noalloc):
    """specdec.bind_step: the step checked and marshalled once, then called on
    new contents of the same buffers, equals the plain call bit for bit."""
    n, W_in, pad_in, cap = wl.initial_geometry(W, 0)
    src0 = wl.make_kv(W, pad_in, W_in, cap, 0, device="cuda")
    s0 = wl.make_token_rows(W, pad_in, W_in, W_in + 2, 0, PAD_ID, device="cuda")
    inputs = [_inputs(t, False) for t in range(4)]
    eager = _Step(sd, variant, False, src0, pad_in, W_in, inputs[0])
    bound = _Step(sd, variant, False, src0, pad_in, W_in, inputs[0])
    b, i = bound.bufs, bound.inp
    call = sd.bind_step(i["logits"], i["draft"], bound.pad, W_in, bound.src, bound.dst, b.tokens, b.n_acc, b.bonus,
                        b.pad_out, b.w_new, b.pos, b.mask, None if noalloc else b.workspace, b.dev_status,
                        s_in=bound.s_in, s_out=bound.s_out, pad_id=PAD_ID, noalloc=noalloc)
    accepted = set()
    for t in (1, 2, 3, 1):
        say(f"bound step variant={variant} noalloc={noalloc} inputs={t}")
        eager.load(inputs[t], src0, s0)
        eager()
        bound.load(inputs[t], src0, s0)
        call()
        torch.cuda.synchronize()
        want, got = eager.result(), bound.result()
        assert want["status"] == 0 and got["status"] == 0
        for name in want:
            assert np.array_equal(np.asarray(got[name]), np.asarray(want[name])), f"inputs {t}: {name} differs"
        accepted.add(tuple(got["n_acc"].tolist()))
    assert len(accepted) > 1


def test_timers_skip_launches_recorded_into_a_graph(sd):
    """With the kernel timers on, a step captured into a graph records no
    timer events; its replays are not counted, the eager steps after them
    are, and the timers keep working."""
    n, W_in, pad_in, cap = wl.initial_geometry(W, 0)
    src0 = wl.make_kv(W, pad_in, W_in, cap, 0, device="cuda")
    s0 = wl.make_token_rows(W, pad_in, W_in, W_in + 2, 0, PAD_ID, device="cuda")
    step = _Step(sd, "oop", False, src0, pad_in, W_in, _inputs(0, False))
    step.load(_inputs(0, False), src0, s0)
    sd.timing_reset()
    sd.timing_enable(sd.TIMING_ALL)
    try:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(3):
            g.replay()
        step()
        step()
        torch.cuda.synchronize()
        say("timers after a captured step")
        for kernel in (sd.KERNEL_VERIFY, sd.KERNEL_REALIGN):
            ms, n_launch = sd.timing_query(kernel)
            assert n_launch == 3 and ms > 0, (kernel, n_launch, ms)   # the warm-up and the two eager steps
    finally:
        sd.timing_enable(False)
        sd.timing_reset()
