"""GPU parity of EXSpec's pool traffic (Algorithm 2) through the C ABI:
batch gather (GetBatch, with fused token rows, paddings and position ids /
mask) and write-back (whole row and append-only), element by element against
the oracle on the same input bytes; device-side range checks; and whole
EXSpec / EqSpec decoding loops over the toy model on the GPU (library
scheduler and kernels) against the same loops on the oracle."""
import numpy as np
import pytest
import torch

import oracle
from oracle.exspec import SequencePool
from tests import exspec_loop as el
from tests.gpu_util import SENT_KV, SENT_MASK, SENT_POS, SENT_TOK, HipBackend, bits, say

pytestmark = pytest.mark.gpu

PAD = -3


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec
    return specdec


def _host_pool(rng, N, L, H, D, cap, lens, tok_stride):
    """Pool with arbitrary 16-bit patterns (NaNs included: the copy is bitwise)
    on [0, len) and 0xFFFF beyond; token rows with -9 beyond len."""
    pool = np.full((L, 2, N, H, cap, D), 0xFFFF, np.uint16)
    tok = np.full((N, tok_stride), -9, np.int32)
    for s in range(N):
        n = int(lens[s])
        pool[:, :, s, :, :n, :] = rng.integers(0, 0x10000, size=(L, 2, H, n, D), dtype=np.uint16)
        tok[s, : n + 1] = rng.integers(0, 50000, size=n + 1)
    return pool, tok


def _dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# (L, H, D, N, B, max len, same length, extra width, k)
GATHER_CASES = [
    (2, 2, 16, 6, 3, 40, False, 0, 4),
    (1, 3, 8, 9, 9, 25, True, 0, 2),        # every slot, same length: plain concatenation
    (2, 2, 128, 12, 5, 300, False, 3, 5),   # spans of several 1024-vector groups, ragged tail
    (1, 1, 256, 4, 4, 150, False, 0, 0),    # k = 0
    (2, 1, 64, 7, 3, 70, True, 5, 7),       # same length, width above the longest row
    (1, 2, 8, 5, 5, 0, False, 2, 3),        # empty sequences only
]


@pytest.mark.parametrize("case", GATHER_CASES, ids=lambda c: f"L{c[0]}H{c[1]}D{c[2]}N{c[3]}B{c[4]}n{c[5]}")
@pytest.mark.parametrize("seed", [0, 1])
def test_gather_matches_oracle(sd, case, seed):
    L, H, D, N, B, nmax, same, extra, k = case
    say(f"gather case={case} seed={seed}")
    rng = np.random.default_rng(100 + seed)
    cap = nmax + 9
    lens = rng.integers(0, nmax + 1, size=N).astype(np.int32)
    if same:
        lens[:] = lens[0]
    elif seed:
        lens[rng.integers(N)] = 0                   # an empty sequence in the batch's pool
    pool, tok = _host_pool(rng, N, L, H, D, cap, lens, cap + 4)
    slots = rng.permutation(N)[:B].astype(np.int32)
    Lb = int(lens[slots].max()) + extra
    bcap, bstride, pm_cap = Lb + k + 1 + 2, Lb + 1 + 3, Lb + k + 1 + 4
    batch = torch.full((L, 2, B, H, bcap, D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    btok = torch.full((B, bstride), SENT_TOK, dtype=torch.int32, device="cuda")
    pads = torch.full((B,), -99, dtype=torch.int32, device="cuda")
    pos = torch.full((B, pm_cap), SENT_POS, dtype=torch.int64, device="cuda")
    mask = torch.full((B, pm_cap), SENT_MASK, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_gather_batch(_dev16(pool), _dev(tok), _dev(lens), _dev(slots), Lb, batch, pads, batch_tok=btok,
                            pos=pos, mask=mask, k=k, pad_id=PAD, dev_status=status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    exp_b = np.full((L, 2, B, H, bcap, D), SENT_KV, np.uint16)
    exp_t = np.full((B, bstride), SENT_TOK, np.int32)
    eb, et, ep = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bstride, PAD, out=(exp_b, exp_t))
    got = bits(batch)
    assert np.array_equal(pads.cpu().numpy(), ep), "paddings differ from the oracle"
    assert np.array_equal(got, eb), "batch cache differs from the oracle (or columns >= Lb were written)"
    assert np.array_equal(btok.cpu().numpy(), et), "batch token rows differ from the oracle"
    epos, emask = oracle.posmask(ep, Lb, k, pm_cap)
    width = Lb + k + 1
    gp, gm = pos.cpu().numpy(), mask.cpu().numpy()
    assert np.array_equal(gp[:, :width], epos[:, :width]) and np.array_equal(gm[:, :width], emask[:, :width])
    assert np.all(gp[:, width:] == SENT_POS) and np.all(gm[:, width:] == SENT_MASK)


def test_gather_without_token_rows_or_posmask(sd):
    rng = np.random.default_rng(5)
    L, H, D, N, B = 2, 2, 16, 5, 3
    lens = np.array([7, 3, 9, 0, 5], np.int32)
    pool, tok = _host_pool(rng, N, L, H, D, 12, lens, 13)
    slots = np.array([4, 3, 2], np.int32)
    batch = torch.full((L, 2, B, H, 10, D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    pads = torch.full((B,), -99, dtype=torch.int32, device="cuda")
    sd.specdec_gather_batch(_dev16(pool), None, _dev(lens), _dev(slots), 9, batch, pads)
    torch.cuda.synchronize()
    eb, _, ep = oracle.gather_batch(pool, tok, lens, slots, 9, 10, 10, PAD,
                                    out=(np.full((L, 2, B, H, 10, D), SENT_KV, np.uint16), np.zeros((B, 10), np.int32)))
    assert np.array_equal(pads.cpu().numpy(), ep) and np.array_equal(bits(batch), eb)


def test_gather_flags_bad_slots(sd):
    """A slot outside [0, N), or one whose length exceeds the width, is skipped
    (pads -1, no byte of its row written) and flagged; other rows are
    gathered."""
    rng = np.random.default_rng(6)
    L, H, D, N, B = 1, 2, 16, 4, 4
    lens = np.array([5, 9, 3, 4], np.int32)
    pool, tok = _host_pool(rng, N, L, H, D, 12, lens, 13)
    slots = np.array([0, 7, 1, 3], np.int32)       # slot 7 does not exist; slot 1 is longer than Lb
    Lb = 6
    batch = torch.full((L, 2, B, H, 8, D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    btok = torch.full((B, 8), SENT_TOK, dtype=torch.int32, device="cuda")
    pads = torch.full((B,), -99, dtype=torch.int32, device="cuda")
    pos = torch.full((B, 10), SENT_POS, dtype=torch.int64, device="cuda")
    mask = torch.full((B, 10), SENT_MASK, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_gather_batch(_dev16(pool), _dev(tok), _dev(lens), _dev(slots), Lb, batch, pads, batch_tok=btok,
                            pos=pos, mask=mask, k=2, pad_id=PAD, dev_status=status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == sd.DEV_BAD_SLOT
    p = pads.cpu().numpy()
    assert p[1] == -1 and p[2] == -1 and p[0] == Lb - 5 and p[3] == Lb - 4
    got = bits(batch)
    for r in (1, 2):
        assert np.all(got[:, :, r] == SENT_KV) and np.all(btok.cpu().numpy()[r] == SENT_TOK)
        assert np.all(pos.cpu().numpy()[r] == SENT_POS) and np.all(mask.cpu().numpy()[r] == SENT_MASK)
    good = np.array([0, 3])
    eb, et, _ = oracle.gather_batch(pool, tok, lens, slots[good], Lb, 8, 8, PAD)
    assert np.array_equal(got[:, :, good, :, :Lb], eb[..., :Lb, :])
    assert np.array_equal(btok.cpu().numpy()[good, : Lb + 1], et[:, : Lb + 1])


def test_gather_split_over_launches(sd, monkeypatch):
    """A grid larger than one dispatch allows is split over launches (forced
    with a tiny cap); the result is unchanged."""
    rng = np.random.default_rng(8)
    L, H, D, N, B = 2, 3, 32, 6, 4
    lens = rng.integers(10, 120, size=N).astype(np.int32)
    pool, tok = _host_pool(rng, N, L, H, D, 128, lens, 130)
    slots = np.array([5, 1, 0, 3], np.int32)
    Lb = int(lens[slots].max())
    outs = []
    for cap_items in (None, 64 * 40):
        if cap_items is None:
            monkeypatch.delenv("SPECDEC_MAX_LAUNCH_ITEMS", raising=False)
        else:
            monkeypatch.setenv("SPECDEC_MAX_LAUNCH_ITEMS", str(cap_items))
        batch = torch.full((L, 2, B, H, Lb + 2, D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        btok = torch.full((B, Lb + 1), SENT_TOK, dtype=torch.int32, device="cuda")
        pads = torch.zeros(B, dtype=torch.int32, device="cuda")
        sd.specdec_gather_batch(_dev16(pool), _dev(tok), _dev(lens), _dev(slots), Lb, batch, pads, batch_tok=btok,
                                pad_id=PAD)
        torch.cuda.synchronize()
        outs.append((bits(batch), btok.cpu().numpy(), pads.cpu().numpy()))
    monkeypatch.delenv("SPECDEC_MAX_LAUNCH_ITEMS", raising=False)
    eb, et, ep = oracle.gather_batch(pool, tok, lens, slots, Lb, Lb + 2, Lb + 1, PAD,
                                     out=(np.full((L, 2, B, H, Lb + 2, D), SENT_KV, np.uint16),
                                          np.full((B, Lb + 1), SENT_TOK, np.int32)))
    for b, t, p in outs:
        assert np.array_equal(b, eb) and np.array_equal(t, et) and np.array_equal(p, ep)


def _writeback_setup(rng, L, H, D, N, B, nmax, k, same=False):
    cap = nmax + k + 2
    lens = rng.integers(0, nmax + 1, size=N).astype(np.int32)
    if same:
        lens[:] = nmax
    pool, tok = _host_pool(rng, N, L, H, D, cap, lens, cap + 2)
    slots = rng.permutation(N)[:B].astype(np.int32)
    Lb = int(lens[slots].max())
    bcap, bstride = Lb + k + 1 + 1, Lb + k + 2 + 2
    batch, btok, pads = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bstride, PAD)
    # the verify window's fresh entries, and garbage in the spare column
    batch[..., Lb:, :] = rng.integers(0, 0x10000, size=batch[..., Lb:, :].shape, dtype=np.uint16)
    tokens = rng.integers(0, 50000, size=(B, k + 1)).astype(np.int32)
    n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
    return pool, tok, lens, slots, Lb, batch, btok, pads, tokens, n_acc


@pytest.mark.parametrize("mode", ["full", "append"])
@pytest.mark.parametrize("case", [(2, 2, 16, 7, 4, 30, 3), (1, 2, 128, 10, 6, 200, 5), (2, 1, 8, 3, 3, 5, 0),
                                  (1, 1, 64, 5, 5, 90, 7)], ids=lambda c: f"L{c[0]}H{c[1]}D{c[2]}N{c[3]}B{c[4]}")
def test_writeback_matches_oracle(sd, case, mode):
    L, H, D, N, B, nmax, k = case
    say(f"write-back case={case} mode={mode}")
    rng = np.random.default_rng(hash((case, mode)) % (1 << 32))
    pool, tok, lens, slots, Lb, batch, btok, pads, tokens, n_acc = _writeback_setup(rng, L, H, D, N, B, nmax, k)
    d_pool, d_tok, d_lens, d_btok = _dev16(pool), _dev(tok), _dev(lens), _dev(btok)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    m = sd.WRITEBACK_FULL if mode == "full" else sd.WRITEBACK_APPEND
    sd.specdec_scatter_accepted(_dev16(batch), _dev(pads), _dev(tokens), _dev(n_acc), _dev(slots), Lb, d_pool, d_tok,
                                d_lens, batch_tok=d_btok, mode=m, dev_status=status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    oracle.scatter_accepted(batch, pads, tokens, n_acc, slots, Lb, pool, tok, lens, batch_tok=btok)
    assert np.array_equal(d_lens.cpu().numpy(), lens), "slot lengths differ from the oracle"
    assert np.array_equal(d_tok.cpu().numpy(), tok), "pool token rows differ from the oracle"
    assert np.array_equal(d_btok.cpu().numpy(), btok), "batch token rows differ from the oracle"
    got = bits(d_pool)
    assert np.array_equal(got, pool), "pool cache differs from the oracle (including columns it must not touch)"


def test_writeback_full_rewrites_changed_rows(sd):
    """The whole-row mode copies every column, also when the batch's content
    no longer equals the slot (the append mode's precondition does not hold)."""
    rng = np.random.default_rng(12)
    pool, tok, lens, slots, Lb, batch, btok, pads, tokens, n_acc = _writeback_setup(rng, 2, 2, 16, 6, 4, 20, 3)
    batch[..., :Lb, :] ^= np.uint16(0x0101)            # content no longer what the slots hold
    d_pool, d_tok, d_lens = _dev16(pool), _dev(tok), _dev(lens)
    sd.specdec_scatter_accepted(_dev16(batch), _dev(pads), _dev(tokens), _dev(n_acc), _dev(slots), Lb, d_pool, d_tok,
                                d_lens, mode=sd.WRITEBACK_FULL)
    torch.cuda.synchronize()
    oracle.scatter_accepted(batch, pads, tokens, n_acc, slots, Lb, pool, tok, lens)
    assert np.array_equal(bits(d_pool), pool) and np.array_equal(d_lens.cpu().numpy(), lens)


def test_writeback_flags_bad_rows(sd):
    """Rows with a slot outside [0, N), n_acc outside [0, k], or a grown length
    above the pool's capacity are skipped and flagged; a length that does not
    match the batch is flagged and still written back."""
    rng = np.random.default_rng(13)
    k = 3
    pool, tok, lens, slots, Lb, batch, btok, pads, tokens, n_acc = _writeback_setup(rng, 1, 2, 16, 8, 5, 12, k)
    slots = slots.copy()
    n_acc = n_acc.copy()
    slots[0] = 99
    n_acc[1] = k + 1
    lens_dev = lens.copy()
    lens_dev[slots[2]] += 1                            # mismatch: flagged, still written
    d_pool, d_tok, d_lens = _dev16(pool), _dev(tok), _dev(lens_dev)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_scatter_accepted(_dev16(batch), _dev(pads), _dev(tokens), _dev(n_acc), _dev(slots), Lb, d_pool, d_tok,
                                d_lens, mode=sd.WRITEBACK_FULL, dev_status=status)
    torch.cuda.synchronize()
    st = int(status.cpu()[0])
    assert st == sd.DEV_BAD_SLOT | sd.DEV_BAD_ACCEPT | sd.DEV_SLOT_LEN
    good = np.array([2, 3, 4])
    exp_pool, exp_tok, exp_lens = pool.copy(), tok.copy(), lens.copy()
    oracle.scatter_accepted(batch[:, :, good], pads[good], tokens[good], n_acc[good], slots[good], Lb, exp_pool,
                            exp_tok, exp_lens)
    assert np.array_equal(bits(d_pool), exp_pool), "a flagged row touched the pool, or a good row differs"
    assert np.array_equal(d_tok.cpu().numpy(), exp_tok)
    assert np.array_equal(d_lens.cpu().numpy(), exp_lens)
    # a pool too small for a grown row
    pool2, tok2, lens2, slots2, Lb2, batch2, btok2, pads2, tokens2, n_acc2 = _writeback_setup(rng, 1, 1, 8, 3, 3, 6, 2,
                                                                                             same=True)
    small = np.ascontiguousarray(pool2[..., : Lb2 + 1, :])
    n_acc2[:] = 2
    d_small, d_tok2, d_lens2 = _dev16(small), _dev(tok2), _dev(lens2)
    status.zero_()
    sd.specdec_scatter_accepted(_dev16(batch2), _dev(pads2), _dev(tokens2), _dev(n_acc2), _dev(slots2), Lb2, d_small,
                                d_tok2, d_lens2, mode=sd.WRITEBACK_APPEND, dev_status=status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) & sd.DEV_BAD_SLOT
    assert np.array_equal(bits(d_small), small), "no row fits: the pool must be unchanged"


def _loop_setup(seed, N, equal_groups):
    rng = np.random.default_rng(seed)
    from tests.toy_model import ToyModel
    model = ToyModel(V=61, n_layers=2, H=2, D=16, accept=0.7, salt=seed)
    prompts = el.random_prompts(rng, N, 3, 40, 61, equal_groups=equal_groups)
    return model, prompts


@pytest.mark.parametrize("mode", ["full", "append"])
@pytest.mark.parametrize("cfg", [(16, 8, 4, 3, 3), (9, 5, 3, 2, 0), (12, 12, 4, 5, 1)],
                         ids=lambda c: f"N{c[0]}W{c[1]}B{c[2]}k{c[3]}g{c[4]}")
def test_exspec_loop_matches_oracle(sd, cfg, mode):
    """Algorithm 2 end to end on the GPU (library scheduler, gather, verify,
    write-back) against the same loop on the oracle: identical schedules,
    generated tokens, pool caches and lengths; and every sequence's output is
    what sequential greedy decoding gives (Corollary B.2)."""
    N, W, B, k, groups = cfg
    say(f"exspec loop cfg={cfg} mode={mode}")
    model, prompts = _loop_setup(50 + N, N, groups)
    max_new = 14
    init = [len(p) - 1 for p in prompts]
    be = HipBackend(writeback=sd.WRITEBACK_FULL if mode == "full" else sd.WRITEBACK_APPEND)
    got = el.run_exspec(be, model, prompts, sd.Scheduler(init, window=W, batch=B, max_new=max_new), k=k,
                        max_new=max_new)
    want = el.run_exspec(el.OracleBackend(), model, prompts, SequencePool(init, window=W, batch=B, max_new=max_new),
                         k=k, max_new=max_new)
    assert got.trace == want.trace, "the schedules differ"
    assert [list(map(int, g)) for g in got.generated] == [list(map(int, g)) for g in want.generated]
    assert np.array_equal(got.lens, want.lens)
    assert np.array_equal(got.pool_tok, want.pool_tok)
    assert np.array_equal(got.pool, want.pool), "pool caches differ"
    el.check_equivalence(model, prompts, got, max_new)
    el.check_pool_cache(model, prompts, got)


def test_eqspec_loop_on_gpu(sd):
    """Algorithm 1 end to end on the GPU (verify, realign of cache and token
    row, position ids / mask): Corollary B.2 over the toy model."""
    model, prompts = _loop_setup(77, 7, 0)
    res = el.run_eqspec(HipBackend(), model, prompts, B=4, k=4, max_new=12)
    el.check_equivalence(model, prompts, res, 12)


def _view_at(nbytes_offset, shape, fill=SENT_KV):
    """A contiguous bf16 tensor of ``shape`` whose data starts ``nbytes_offset``
    bytes past a 16 KB boundary (a view into a larger buffer)."""
    n = int(np.prod(shape))
    buf = torch.full((n + 3 * 8192,), fill, dtype=torch.int16, device="cuda")
    base = buf.data_ptr()
    skip = ((-base) % 16384 + nbytes_offset) // 2
    return buf[skip: skip + n].view(shape).view(torch.bfloat16)


OFFSETS = [0, 256, 1024, 4096 + 256, 16384 - 256]


@pytest.mark.parametrize("offset", OFFSETS)
@pytest.mark.parametrize("cap_kind", ["aligned", "ragged"])
def test_alignment_of_destination(sd, offset, cap_kind):
    """Gather, whole-row write-back and out-of-place realignment with the
    destination at various offsets from a 16 KB boundary and capacities that
    are (or are not) a multiple of 16 KB per span: the spans are tiled from the
    group boundary below them when they are not aligned; results equal the
    oracle's, and nothing outside the written columns changes."""
    say(f"alignment offset={offset} cap={cap_kind}")
    rng = np.random.default_rng(offset + (0 if cap_kind == "aligned" else 1))
    L, H, D, N, B, k = 1, 2, 128, 6, 4, 3             # 16 vectors per column: 64 columns = 16 KB
    lens = rng.integers(40, 140, size=N).astype(np.int32)
    pcap = 192 if cap_kind == "aligned" else 171
    pool, tok = _host_pool(rng, N, L, H, D, pcap, lens, pcap + 2)
    slots = rng.permutation(N)[:B].astype(np.int32)
    Lb = int(lens[slots].max())
    bcap = 192 if cap_kind == "aligned" else Lb + k + 1
    batch = _view_at(offset, (L, 2, B, H, bcap, D))
    pads = torch.zeros(B, dtype=torch.int32, device="cuda")
    btok = torch.full((B, bcap + 1), SENT_TOK, dtype=torch.int32, device="cuda")
    sd.specdec_gather_batch(_dev16(pool), _dev(tok), _dev(lens), _dev(slots), Lb, batch, pads, batch_tok=btok,
                            pad_id=PAD)
    torch.cuda.synchronize()
    eb, et, ep = oracle.gather_batch(pool, tok, lens, slots, Lb, bcap, bcap + 1, PAD,
                                     out=(np.full((L, 2, B, H, bcap, D), SENT_KV, np.uint16),
                                          np.full((B, bcap + 1), SENT_TOK, np.int32)))
    assert np.array_equal(bits(batch), eb), "gather differs from the oracle"
    # write-back (whole rows) into a pool placed at the same offset
    dpool = _view_at(offset, pool.shape)
    dpool.view(torch.int16).copy_(torch.from_numpy(pool.view(np.int16)).cuda())
    hb = bits(batch)
    hb[..., Lb:, :] = rng.integers(0, 0x10000, size=hb[..., Lb:, :].shape, dtype=np.uint16)
    batch.view(torch.int16).copy_(torch.from_numpy(hb.view(np.int16)).cuda())
    tokens = rng.integers(0, 999, size=(B, k + 1)).astype(np.int32)
    n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
    d_tok, d_lens = _dev(tok), _dev(lens)
    sd.specdec_scatter_accepted(batch, pads, _dev(tokens), _dev(n_acc), _dev(slots), Lb, dpool, d_tok, d_lens,
                                mode=sd.WRITEBACK_FULL)
    torch.cuda.synchronize()
    exp_pool, exp_tok, exp_lens = pool.copy(), tok.copy(), lens.copy()
    oracle.scatter_accepted(hb, ep, tokens, n_acc, slots, Lb, exp_pool, exp_tok, exp_lens)
    assert np.array_equal(bits(dpool), exp_pool), "write-back differs from the oracle"
    assert np.array_equal(d_lens.cpu().numpy(), exp_lens)
    # out-of-place realignment of the batch into a destination at the offset
    W_in = Lb + k + 1
    dst = _view_at(offset, (L, 2, B, H, bcap, D))
    w_new = int((Lb - ep + n_acc + 1).max())
    sd.specdec_realign_kv(batch, dst, k, W_in, pads, _dev(n_acc),
                          torch.tensor([w_new], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    exp = oracle.realign_kv(hb, k, W_in, ep, n_acc, w_new, dst=np.full(hb.shape, SENT_KV, np.uint16))
    assert np.array_equal(bits(dst), exp), "realignment differs from the oracle"
