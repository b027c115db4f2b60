"""Concurrent calls: the library keeps no state between calls but the kernel
timers (behind a mutex) and the thread-local error text, so steps issued
from several host threads, each on its own stream with its own buffers, give
the results of the same steps run one after another.  Each thread also makes
a call that fails validation, and must read its own error text back."""
import threading

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


class _Job:
    def __init__(self, sd, seed, stream, tag):
        self.sd, self.stream, self.tag = sd, stream, tag
        n, self.W_in, self.pad_in, cap = wl.initial_geometry(W, seed)
        self.src = wl.make_kv(W, self.pad_in, self.W_in, cap, seed, device="cuda")
        self.dst = torch.empty_like(self.src)
        self.steps = [wl.logits_and_drafts(W, seed, t, device="cuda")[:2] for t in range(6)]
        self.pad = torch.as_tensor(self.pad_in, device="cuda")
        self.bufs = sd.StepBuffers(W.B, W.k, W.V, self.W_in + W.k + 1)
        self.s_in = wl.make_token_rows(W, self.pad_in, self.W_in, self.W_in + 2, seed, PAD_ID, device="cuda")
        self.s_out = torch.empty_like(self.s_in)
        self.results = []
        self.error_text = None

    def run(self):
        with torch.cuda.stream(self.stream):
            for lg, dr in self.steps:
                b = self.bufs
                self.sd.specdec_step(lg, dr, self.pad, self.W_in, self.src, self.dst, b.tokens, b.n_acc, b.bonus,
                                     b.pad_out, b.w_new, b.pos, b.mask, b.workspace, b.dev_status,
                                     s_in=self.s_in, s_out=self.s_out, pad_id=PAD_ID, stream=self.stream)
                self.stream.synchronize()
                w = int(b.w_new.cpu()[0])
                width = w + W.k + 1                # the columns the step writes
                self.results.append(dict(tokens=b.tokens.cpu().numpy(), n_acc=b.n_acc.cpu().numpy(),
                                         pad_out=b.pad_out.cpu().numpy(), w=w, pos=b.pos.cpu().numpy()[:, :width],
                                         mask=b.mask.cpu().numpy()[:, :width], kv=bits(self.dst[..., :w, :]),
                                         s=self.s_out.cpu().numpy()[:, :w + 1], status=int(b.dev_status.cpu()[0])))
            # a call that fails validation: the error text is this thread's own
            rc = self.sd.lib.specdec_build_posmask(None, None, W.B, W.k, None, None, self.tag, None, None)
            self.error_text = (rc, self.sd.lib.specdec_last_error().decode())


def test_concurrent_streams_match_sequential(sd):
    sd.timing_enable(True)                  # the timers' queue is shared by the threads
    streams = [torch.cuda.Stream() for _ in range(3)]
    seq = [_Job(sd, 10 + j, streams[j], j + 1) for j in range(3)]
    for job in seq:
        job.run()
    par = [_Job(sd, 10 + j, streams[j], j + 1) for j in range(3)]
    torch.cuda.synchronize()
    threads = [threading.Thread(target=job.run) for job in par]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    sd.timing_enable(False)
    total_ms, launches = sd.timing_query(sd.KERNEL_REALIGN)
    assert launches >= 36 and total_ms > 0
    sd.timing_reset()
    for j, (a, b) in enumerate(zip(seq, par)):
        say(f"stream job {j}: {len(b.results)} steps")
        assert len(a.results) == len(b.results) == 6
        for ra, rb in zip(a.results, b.results):
            assert ra["status"] == 0 and rb["status"] == 0
            for name in ra:
                assert np.array_equal(np.asarray(ra[name]), np.asarray(rb[name])), f"job {j}: {name} differs"
        rc, text = b.error_text
        assert rc == 1 and f"pm_cap={j + 1} " in text, text      # pm_cap below k+1, named in this thread's text
