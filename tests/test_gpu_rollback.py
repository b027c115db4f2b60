"""GPU parity of the two rollback strategies (Section 2, Family A and
Family B) through the C ABI against the oracle, bit-exact: Family A's
truncation to the batch-minimum accepted count (with the in-place
realignment that then moves nothing, and a whole rollback decoding loop over
the toy model), and Family B's compaction of a flat variable-length cache
with its cumulative offsets and position ids."""
import numpy as np
import pytest
import torch

import oracle
from tests import exspec_loop as el
from tests.gpu_util import SENT_KV, HipBackend, bits, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec
    return specdec


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _rollback(sd, tokens, n_acc, pad, W_in, in_place=False):
    B = len(n_acc)
    i32 = dict(dtype=torch.int32, device="cuda")
    t, na, pd = _dev(tokens), _dev(n_acc), _dev(pad)
    out = dict(n_acc=na if in_place else torch.full((B,), -9, **i32), bonus=torch.full((B,), -9, **i32),
               pad_out=pd if in_place else torch.full((B,), -9, **i32), w_new=torch.full((1,), -9, **i32))
    st = torch.zeros(1, **i32)
    sd.specdec_rollback(t, na, pd, W_in, out["n_acc"], out["bonus"], out["pad_out"], out["w_new"], st)
    torch.cuda.synchronize()
    res = {n: v.cpu().numpy() for n, v in out.items()}
    res["w_new"] = int(res["w_new"][0])
    res["status"] = int(st.cpu()[0])
    return res


@pytest.mark.parametrize("B,k,L", [(1, 4, 10), (8, 5, 1018), (64, 4, 300), (2048, 7, 40), (5, 0, 3), (3, 64, 70)])
@pytest.mark.parametrize("in_place", [False, True])
def test_rollback_matches_oracle(sd, B, k, L, in_place):
    rng = np.random.default_rng(B * 100 + k)
    W_in = L + k + 1
    tokens = rng.integers(0, 50000, size=(B, k + 1)).astype(np.int32)
    n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
    pad = rng.integers(0, L + 1, size=B).astype(np.int32)
    if B > 2:
        pad[1] = 0
    got = _rollback(sd, tokens, n_acc, pad, W_in, in_place)
    want = oracle.rollback(tokens, n_acc, pad, W_in)
    assert got["status"] == 0
    for name in ("n_acc", "bonus", "pad_out"):
        assert np.array_equal(got[name], want[name]), name
    assert got["w_new"] == want["w_new"]


def test_rollback_flags_bad_rows(sd):
    rng = np.random.default_rng(3)
    B, k, L = 6, 3, 12
    tokens = rng.integers(0, 99, size=(B, k + 1)).astype(np.int32)
    n_acc = np.array([2, 3, 9, 1, 2, 3], np.int32)    # row 2: n_acc out of range
    pad = np.array([0, 4, 1, 2, 13, 3], np.int32)     # row 4: pad out of range
    got = _rollback(sd, tokens, n_acc, pad, L + k + 1)
    assert got["status"] == sd.DEV_BAD_ACCEPT | sd.DEV_BAD_PAD_IN
    good = np.array([0, 1, 3, 5])
    want = oracle.rollback(tokens[good], n_acc[good], pad[good], L + k + 1)
    assert np.array_equal(got["n_acc"][good], want["n_acc"]) and got["w_new"] == want["w_new"]
    assert np.array_equal(got["pad_out"][good], want["pad_out"]) and got["pad_out"][2] == -1 and got["pad_out"][4] == -1


def test_rollback_then_realign_in_place_moves_nothing(sd):
    """After a rollback with minimum padding 0 every offset is zero: the
    in-place realignment leaves the cache bit for bit as it was, and the
    out-of-place one equals the oracle's."""
    from paper_2510_22876_amd import workloads as wl
    w = wl.WORKLOADS["vicuna7b"].scaled(L=4, H=8)
    n, W_in, pad_in, cap = wl.initial_geometry(w)
    logits, draft, *_ = wl.logits_and_drafts(w, 0, 0, device="cuda")
    v = oracle.verify(logits.cpu(), w.logit_dtype, draft.cpu().numpy(), pad_in, W_in)
    r = oracle.rollback(v["tokens"], v["n_acc"], pad_in, W_in)
    assert np.array_equal(r["pad_out"], pad_in)
    kv = wl.make_kv(w, pad_in, W_in, cap, device="cuda")
    before = kv.clone()
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_realign_kv(kv, kv, w.k, W_in, _dev(pad_in), _dev(r["n_acc"]), _dev(np.array([r["w_new"]], np.int32)), st)
    torch.cuda.synchronize()
    assert int(st.cpu()[0]) == 0
    assert torch.equal(kv.view(torch.int16), before.view(torch.int16))
    dst = torch.zeros_like(kv)
    sd.specdec_realign_kv(kv, dst, w.k, W_in, _dev(pad_in), _dev(r["n_acc"]), _dev(np.array([r["w_new"]], np.int32)))
    exp = oracle.realign_kv(bits(before), w.k, W_in, pad_in, r["n_acc"], r["w_new"])
    W = r["w_new"]
    assert np.array_equal(bits(dst)[..., :W, :], exp[..., :W, :])


def test_rollback_loop_on_gpu(sd):
    """A rollback decoding loop on the GPU (verify, rollback, realign) equals
    the oracle's loop round by round and generates sequential greedy output."""
    from tests.toy_model import ToyModel
    rng = np.random.default_rng(5)
    model = ToyModel(V=61, n_layers=2, H=2, D=16, accept=0.7, salt=5)
    prompts = el.random_prompts(rng, 6, 3, 30, 61)
    got = el.run_eqspec(HipBackend(), model, prompts, B=3, k=4, max_new=12, rollback=True)
    want = el.run_eqspec(el.OracleBackend(), model, prompts, B=3, k=4, max_new=12, rollback=True)
    assert got.trace == want.trace and got.generated == want.generated
    el.check_equivalence(model, prompts, got, 12)


def _varlen(rng, B, k, L, H, D, cmax=40, extra=7):
    c = rng.integers(0, cmax + 1, size=B)
    lens = c + k + 1
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1]) + extra
    src = rng.integers(0, 0x10000, size=(L, 2, T, H, D), dtype=np.uint16)
    n_acc = rng.integers(0, k + 1, size=B).astype(np.int32)
    return cu, src, n_acc, T, int(lens.max())


def _run_varlen(sd, src, cu, n_acc, k, max_len, dst_T=None, status=None):
    L, _, T, H, D = src.shape
    s = torch.from_numpy(src.view(np.int16)).cuda().view(torch.bfloat16)
    d = torch.full((L, 2, dst_T or T, H, D), SENT_KV, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    B = len(n_acc)
    cu_out = torch.full((B + 1,), -9, dtype=torch.int32, device="cuda")
    pos = torch.full((dst_T or T,), -1, dtype=torch.int64, device="cuda")
    sd.specdec_varlen_rollback(s, d, _dev(cu), _dev(n_acc), k, max_len, cu_out, pos, status)
    torch.cuda.synchronize()
    return bits(d), cu_out.cpu().numpy(), pos.cpu().numpy()


# (B, k, L, H, D): rows of 16 B (H*D = 8) to 8 KB (32 x 128)
VARLEN_CASES = [(3, 4, 2, 1, 8), (8, 5, 2, 32, 128), (64, 4, 1, 4, 128), (16, 7, 2, 2, 16), (1, 0, 1, 1, 8),
                (200, 2, 1, 1, 64)]


@pytest.mark.parametrize("case", VARLEN_CASES, ids=lambda c: "B{}k{}L{}H{}D{}".format(*c))
@pytest.mark.parametrize("slack", [0, 50])
def test_varlen_rollback_matches_oracle(sd, case, slack):
    B, k, L, H, D = case
    say(f"varlen case={case} slack={slack}")
    rng = np.random.default_rng(B + k + slack)
    cu, src, n_acc, T, max_len = _varlen(rng, B, k, L, H, D)
    got, cu_out, pos = _run_varlen(sd, src, cu, n_acc, k, max_len + slack, dst_T=T + 3)
    exp_dst = np.full((L, 2, T + 3, H, D), SENT_KV, np.uint16)
    exp, ecu, epos = oracle.varlen_rollback(np.concatenate([src, np.zeros((L, 2, 3, H, D), np.uint16)], axis=2), cu,
                                            n_acc, k, dst=exp_dst)
    assert np.array_equal(cu_out, ecu), "offsets differ from the oracle"
    assert np.array_equal(got, exp), "compacted cache differs from the oracle (or rows beyond were written)"
    assert np.array_equal(pos, epos), "position ids differ from the oracle"


def test_varlen_rollback_flags_bad_segments(sd):
    rng = np.random.default_rng(9)
    B, k, L, H, D = 5, 3, 1, 2, 8
    cu, src, n_acc, T, max_len = _varlen(rng, B, k, L, H, D)
    n_acc = n_acc.copy()
    n_acc[1] = k + 2                                 # out of range
    cu2 = cu.copy()
    cu2[3] = cu2[2] + 2                              # sequence 2 shorter than k + 1
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    got, cu_out, pos = _run_varlen(sd, src, cu2, n_acc, k, T, status=st)
    assert int(st.cpu()[0]) == sd.DEV_BAD_ACCEPT | sd.DEV_BAD_WIDTH
    keep = np.diff(cu_out)
    assert keep[1] == 0 and keep[2] == 0
    for i in (0, 3, 4):
        seg = src[:, :, cu2[i]: cu2[i] + keep[i]]
        assert keep[i] == (cu2[i + 1] - cu2[i]) - (k - n_acc[i])
        assert np.array_equal(got[:, :, cu_out[i]: cu_out[i + 1]], seg)


def test_varlen_rollback_split_over_launches(sd, monkeypatch):
    rng = np.random.default_rng(11)
    cu, src, n_acc, T, max_len = _varlen(rng, 12, 3, 2, 2, 16, cmax=100)
    monkeypatch.setenv("SPECDEC_MAX_LAUNCH_ITEMS", str(64 * 200))
    got, cu_out, pos = _run_varlen(sd, src, cu, n_acc, 3, max_len)
    monkeypatch.delenv("SPECDEC_MAX_LAUNCH_ITEMS")
    exp, ecu, epos = oracle.varlen_rollback(src, cu, n_acc, 3, dst=np.full_like(src, SENT_KV))
    assert np.array_equal(got, exp) and np.array_equal(cu_out, ecu) and np.array_equal(pos, epos)


def test_varlen_rollback_full_size(sd):
    """The vicuna7b shape as a flat cache (8 sequences of U[128,1024] cached
    entries plus 6 window rows, 32 layers, 32 heads of 128): offsets and
    positions against the oracle in full, every sequence's rows with torch on
    the device against the compaction rule, sampled rows against the oracle."""
    from paper_2510_22876_amd import workloads as wl
    w = wl.WORKLOADS["vicuna7b"]
    n = wl.prompt_lengths(w, 0)
    rng = np.random.default_rng(0)
    k = w.k
    lens = n + k + 1
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    n_acc = rng.integers(0, k + 1, size=w.B).astype(np.int32)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    src = torch.randn((w.L, 2, T, w.H, w.D), generator=g, device="cuda").to(torch.bfloat16)
    dst = torch.zeros_like(src)
    cu_out = torch.zeros(w.B + 1, dtype=torch.int32, device="cuda")
    pos = torch.full((T,), -1, dtype=torch.int64, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sd.specdec_varlen_rollback(src, dst, _dev(cu), _dev(n_acc), k, int(lens.max()), cu_out, pos, st)
    torch.cuda.synchronize()
    assert int(st.cpu()[0]) == 0
    co = cu_out.cpu().numpy()
    keep = lens - (k - n_acc)
    assert np.array_equal(co, np.concatenate([[0], np.cumsum(keep)]))
    p = pos.cpu().numpy()
    assert np.array_equal(p[: co[-1]], np.concatenate([np.arange(x) for x in keep])) and np.all(p[co[-1]:] == -1)
    for i in range(w.B):
        assert torch.equal(dst[:, :, co[i]: co[i + 1]].view(torch.int16), src[:, :, cu[i]: cu[i] + keep[i]].view(torch.int16))
    # sampled layers against the oracle
    for l in (0, w.L - 1):
        s1 = bits(src[l:l + 1])
        e, _, _ = oracle.varlen_rollback(s1, cu, n_acc, k)
        assert np.array_equal(bits(dst[l:l + 1])[:, :, : co[-1]], e[:, :, : co[-1]])
