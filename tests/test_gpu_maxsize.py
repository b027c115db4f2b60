"""GPU parity at the limits of the index arithmetic.

* Verification over a vocabulary of 2^31 - 1 bf16 logits: the second logit
  row starts 4.3 GB in, and token indices reach the largest int32.  Expected
  tokens come from the construction: the logits are uniform in [-1, 1] and the
  planted maxima (with ties) are larger, so the answer is the lowest planted
  index (Alg. 3's argmax with the lowest-index tie-break).
* The out-of-place realignment of two 72 GB caches (D = 4096, W_in = 2.2 M
  columns): span offsets reach 4.6 G 16-byte vectors.  Checked with torch on
  the device against the relocation definition (pads +0.0, content = the kept
  source columns bit for bit).
* The in-place realignment of one 138 GB cache whose spans hold 2.15 G
  vectors: the moving row's kept entries lie at vector offsets past 2^31
  within their spans; checked against a copy of them taken before the step.
* Family B compaction of a flat cache of 2^31 - 8 rows.
Caches are compared as int16 bit patterns (random bits include NaNs).
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _free():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec  # noqa: F401
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_verify_largest_vocabulary():
    from paper_2510_22876_amd import specdec as sd
    V = 2**31 - 1
    B, k, W_in = 1, 1, 10
    say(f"verify V={V} bf16: {2 * V * 2 / 1e9:.1f} GB of logits")
    g = torch.Generator(device="cuda")
    g.manual_seed(31)
    logits = torch.empty((B, k + 1, V), dtype=torch.bfloat16, device="cuda")
    logits.uniform_(-1.0, 1.0, generator=g)
    # slot 0: equal maxima at V-5 and V-1; slot 1: equal maxima at 1 and V-2
    logits[0, 0, V - 5] = 2.0
    logits[0, 0, V - 1] = 2.0
    logits[0, 1, 1] = 3.0
    logits[0, 1, V - 2] = 3.0
    i32 = dict(dtype=torch.int32, device="cuda")
    draft = torch.tensor([[V - 5]], **i32)
    pad_in = torch.zeros(B, **i32)
    tokens, n_acc, bonus, pad_out = (torch.full(s, -9, **i32) for s in ((B, k + 1), (B,), (B,), (B,)))
    w_new = torch.full((1,), -9, **i32)
    status = torch.zeros(1, **i32)
    ws = sd.alloc_workspace(B, k, V)
    sd.specdec_verify_greedy(logits, draft, pad_in, W_in, tokens, n_acc, bonus, pad_out, w_new, ws, status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    assert tokens.cpu().tolist() == [[V - 5, 1]]
    assert n_acc.cpu().tolist() == [1] and bonus.cpu().tolist() == [1]
    # Eq. (1)/(2): c = W_in - (k+1) = 8, len = 8 + 1 + 1 = 10 = L', pad_out = 0
    assert int(w_new.cpu()[0]) == 10 and pad_out.cpu().tolist() == [0]
    # a rejected draft on the same logits: the first slot's token is emitted
    draft.fill_(V - 1)
    sd.specdec_verify_greedy(logits, draft, pad_in, W_in, tokens, n_acc, bonus, pad_out, w_new, ws, status)
    torch.cuda.synchronize()
    assert n_acc.cpu().tolist() == [0] and bonus.cpu().tolist() == [V - 5]
    assert int(w_new.cpu()[0]) == 9 and int(status.cpu()[0]) == 0


def _two_rows(W_in, pad1, k=1, V=64):
    """Logits and drafts for two rows: row 0 (padding 0) accepts its draft,
    row 1 (padding pad1) rejects it; so L' = W_in and row 1 shifts by +1."""
    lg = torch.randn((2, k + 1, V), generator=torch.Generator().manual_seed(3))
    lg[0, 0, 17] = 50.0
    lg[1, 0, 23] = 50.0
    draft = torch.tensor([[17], [24]], dtype=torch.int32)
    pad_in = np.array([0, pad1], np.int32)
    v = oracle.verify(lg, "f32", draft.numpy(), pad_in, W_in)
    assert v["n_acc"].tolist() == [1, 0] and v["w_new"] == W_in
    assert v["pad_out"].tolist() == [0, pad1 + 1]
    return lg, draft, pad_in, v


def _step(sd, lg, draft, pad_in, W_in, src, dst, k=1):
    pm_cap = W_in + k + 1
    bufs = sd.StepBuffers(2, k, lg.shape[2], pm_cap)
    dev = lambda a: torch.as_tensor(np.asarray(a), device="cuda")
    sd.specdec_step(dev(lg), dev(draft), dev(pad_in), W_in, src, dst, bufs.tokens, bufs.n_acc, bufs.bonus,
                    bufs.pad_out, bufs.w_new, bufs.pos, bufs.mask, bufs.workspace, bufs.dev_status)
    torch.cuda.synchronize()
    assert int(bufs.dev_status.cpu()[0]) == 0
    return bufs, pm_cap


def _random_cache(cap, D, pad_in):
    src = torch.empty((1, 2, 2, 1, cap, D), dtype=torch.bfloat16, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    src.view(torch.int16).random_(-32768, 32767, generator=g)
    for i, p in enumerate(pad_in):
        src[:, :, i, :, :int(p), :] = 0.0      # input pads are +0.0 (in place needs it)
    return src


def test_realign_out_of_place_beyond_2_32_vectors():
    """Two caches of 72 GB: span offsets reach 4.6 G 16-byte vectors."""
    from paper_2510_22876_amd import specdec as sd
    D, k, W_in = 4096, 1, 2_200_000
    lg, draft, pad_in, v = _two_rows(W_in, 100)
    src = _random_cache(W_in, D, pad_in)
    assert src.numel() // 8 > 2**32
    say(f"out-of-place realign D={D} W_in={W_in}: {src.numel() * 2 / 1e9:.1f} GB per cache")
    dst = torch.empty_like(src)
    bufs, pm_cap = _step(sd, lg, draft, pad_in, W_in, src, dst)
    assert bufs.n_acc.cpu().tolist() == [1, 0] and bufs.pad_out.cpu().tolist() == v["pad_out"].tolist()
    assert int(bufs.w_new.cpu()[0]) == W_in
    pos, mask = oracle.posmask(v["pad_out"], W_in, k, pm_cap)
    assert np.array_equal(bufs.pos.cpu().numpy(), pos) and np.array_equal(bufs.mask.cpu().numpy(), mask)
    lens = (W_in - (k + 1) - pad_in) + v["n_acc"] + 1
    for i in range(2):
        p, q, n = int(pad_in[i]), int(v["pad_out"][i]), int(lens[i])
        for kv in range(2):
            got = dst[0, kv, i, 0].view(torch.int16)
            assert torch.equal(got[q:q + n], src[0, kv, i, 0, p:p + n].view(torch.int16)), f"row {i} kv {kv}"
            if q:
                assert not bool(got[:q].any()), f"row {i} kv {kv}: pads not +0.0"


def test_realign_in_place_beyond_2_31_vectors_per_span():
    """One cache of 138 GB whose spans hold 2.15 G vectors: the moving row's
    kept entries sit at vector offsets past 2^31 within its spans."""
    from paper_2510_22876_amd import specdec as sd
    D, k, W_in = 4096, 1, 4_200_000
    assert W_in * D // 8 > 2**31
    pad1 = W_in - (k + 1) - 1000           # row 1: 1000 cached entries at the far end of its spans
    assert pad1 * D // 8 > 2**31
    lg, draft, pad_in, v = _two_rows(W_in, pad1)
    src = _random_cache(W_in, D, pad_in)
    say(f"in-place realign D={D} W_in={W_in}: {src.numel() * 2 / 1e9:.1f} GB")
    n = 1001                                # row 1 keeps its 1000 entries and the pending one
    ref = [src[0, kv, 1, 0, pad1:pad1 + n].clone() for kv in range(2)]
    untouched = [src[0, kv, 0, 0, W_in - 4:W_in].clone() for kv in range(2)]
    bufs, _ = _step(sd, lg, draft, pad_in, W_in, src, src)
    assert bufs.pad_out.cpu().tolist() == [0, pad1 + 1] and int(bufs.w_new.cpu()[0]) == W_in
    for kv in range(2):
        got = src[0, kv, 1, 0].view(torch.int16)
        assert torch.equal(got[pad1 + 1:pad1 + 1 + n], ref[kv].view(torch.int16)), f"kv {kv}: content differs"
        assert not bool(got[:pad1 + 1].any()), f"kv {kv}: pads not +0.0"
        # row 0 does not move (its padding stays 0)
        assert torch.equal(src[0, kv, 0, 0, W_in - 4:W_in].view(torch.int16), untouched[kv].view(torch.int16))


def test_varlen_rollback_largest_buffer():
    """Family B compaction of a flat cache of 2^31 - 8 rows (two 69 GB
    buffers): row offsets, positions and slab offsets near the int32 limit.
    Checked with torch on the device against the definition (each sequence's
    kept rows moved to the running offset, positions 0..keep-1)."""
    from paper_2510_22876_amd import specdec as sd
    T, k = 2**31 - 8, 1
    src = torch.empty((1, 2, T, 1, 8), dtype=torch.bfloat16, device="cuda")
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    src.view(torch.int16).random_(-32768, 32767, generator=g)
    say(f"varlen rollback T={T}: {src.numel() * 2 / 1e9:.1f} GB per buffer")
    dst = torch.empty_like(src)
    i32 = dict(dtype=torch.int32, device="cuda")
    b1 = 1_200_000_000
    cu_in = torch.tensor([0, b1, T - 3], **i32)
    n_acc = torch.tensor([1, 0], **i32)                 # sequence 0 keeps all its rows, sequence 1 drops one
    keep = [b1, (T - 3 - b1) - 1]
    cu_out = torch.full((3,), -9, **i32)
    pos = torch.full((T,), -1, dtype=torch.int64, device="cuda")
    status = torch.zeros(1, **i32)
    sd.specdec_varlen_rollback(src, dst, cu_in, n_acc, k, b1, cu_out, pos, status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    assert cu_out.cpu().tolist() == [0, keep[0], keep[0] + keep[1]]
    starts = [0, b1]
    o = 0
    for i in range(2):
        for kv in range(2):
            got = dst[0, kv, o:o + keep[i]].view(torch.int16)
            want = src[0, kv, starts[i]:starts[i] + keep[i]].view(torch.int16)
            assert torch.equal(got, want), f"sequence {i} kv {kv}: rows differ"
        assert torch.equal(pos[o:o + keep[i]], torch.arange(keep[i], dtype=torch.int64, device="cuda")), \
            f"sequence {i}: positions"
        o += keep[i]
    assert bool((pos[o:] == -1).all()), "positions written beyond the kept rows"
