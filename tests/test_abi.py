"""The C-ABI library loads, exports every function include/specdec.h declares,
and rejects bad arguments on the host before anything reaches a GPU.

No compute call is made here.  The error-path cases pass dummy pointer values
that the library never dereferences, because each case fails validation; they
are skipped when a GPU is visible, so that a validation regression can never
send such a pointer to a kernel.
"""
import ctypes
import re
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
HEADER = (ROOT / "include" / "specdec.h").read_text()


def _declared_functions():
    body = re.sub(r"/\*.*?\*/", "", HEADER, flags=re.S)
    return sorted(set(re.findall(r"\b(specdec_\w+)\s*\(", body)))


@pytest.fixture(scope="module")
def sd():
    from paper_2510_22876_amd import specdec
    return specdec


def test_library_exports_every_declared_function(sd):
    declared = _declared_functions()
    assert "specdec_step" in declared and "specdec_verify_greedy" in declared
    assert "specdec_realign_kv" in declared and "specdec_build_posmask" in declared
    for name in declared:
        assert hasattr(sd.lib, name), f"{name} declared in specdec.h but not exported"
    assert sorted(sd.EXPORTED) == declared


def test_abi_version_matches_header(sd):
    m = re.search(r"#define SPECDEC_ABI_VERSION (\d+)", HEADER)
    assert sd.abi_version() == int(m.group(1))


def test_workspace_bytes(sd):
    # 48 rows of 32000: 16 workgroups of 2048 elements per row; then the
    # in-place order table (4 words per row)
    assert sd.workspace_bytes(8, 5, 32000) == 256 + 8 * 6 * 16 * 8 + 16 * 8
    assert sd.workspace_bytes(0, 0, 10) == 256
    assert sd.workspace_bytes(-1, 2, 10) == 0
    assert sd.workspace_bytes(4, 65, 10) == 0
    assert sd.workspace_bytes(4, 2, 0) == 0
    # never more than 64 workgroups per row
    assert sd.workspace_bytes(1, 0, 2 ** 31 - 1) == 256 + 64 * 8 + 16


def _no_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("error paths with dummy pointers run on CPU-only hosts")


# A dummy, well-aligned address; never dereferenced (every case fails validation).
A = 0x10000
P = ctypes.c_void_p


def _a(i):
    """Distinct dummy addresses, 16 MiB apart (buffers must not overlap)."""
    return A + ((i + 1) << 24)


LG, DR, PI, TK, NA, BO, PO, WN, WS, POS, MSK, DL, UA, US = (_a(i) for i in range(14))


def _verify(sd, **over):
    args = dict(logits=LG, dtype=1, draft=DR, pad_in=PI, B=2, k=3, V=100, W_in=10, tokens=TK, n_acc=NA,
                bonus=BO, pad_out=PO, w_new=WN, ws=WS, ws_bytes=sd.workspace_bytes(2, 3, 100), status=None,
                stream=None)
    args.update(over)
    return sd.lib.specdec_verify_greedy(*args.values())


@pytest.mark.parametrize("over,code", [
    (dict(B=-1), 1), (dict(B=70000), 1), (dict(k=-1), 1), (dict(k=65), 1), (dict(V=0), 1),
    (dict(W_in=3), 1), (dict(W_in=1 << 25), 1), (dict(dtype=7), 2), (dict(logits=None), 1),
    (dict(draft=None), 1), (dict(pad_in=None), 1), (dict(tokens=None), 1), (dict(n_acc=None), 1),
    (dict(pad_out=None), 1), (dict(w_new=None), 1), (dict(logits=LG + 1), 2), (dict(dtype=0, logits=LG + 2), 2),
    (dict(tokens=TK + 2), 2), (dict(ws=None), 4), (dict(ws=WS + 4), 4), (dict(ws_bytes=16), 4),
    (dict(B=65536, k=63), 1),
    # outputs overlapping inputs or each other (a decode loop passing pad_in as pad_out)
    (dict(pad_out=PI), 1), (dict(n_acc=TK + 4), 1), (dict(tokens=DR), 1), (dict(w_new=PO + 4), 1),
    (dict(ws=LG + 64), 1), (dict(bonus=NA), 1),
])
def test_verify_rejects(sd, over, code):
    _no_gpu()
    assert _verify(sd, **over) == code
    assert sd.lib.specdec_last_error().decode() != ""


def test_verify_empty_batch_is_a_noop(sd):
    _no_gpu()
    assert _verify(sd, B=0, logits=None, draft=None, pad_in=None, tokens=None, n_acc=None, pad_out=None,
                   w_new=None, ws=None) == 0


def _kv(sd, data=A, L=2, B=2, H=2, D=16, cap=64):
    return sd.KV(data, L, B, H, D, cap)


def _realign(sd, src=None, dst=None, k=3, W_in=10, pad_in=A, n_acc=A, w_new=A):
    src = src if src is not None else _kv(sd)
    dst = dst if dst is not None else _kv(sd, data=A + (1 << 30))
    return sd.lib.specdec_realign_kv(ctypes.byref(src), ctypes.byref(dst), k, W_in, pad_in, n_acc, w_new,
                                     None, None)


def test_realign_rejects(sd):
    _no_gpu()
    K = lambda **kw: _kv(sd, **kw)
    assert sd.lib.specdec_realign_kv(None, ctypes.byref(K()), 3, 10, A, A, A, None, None) == 1
    assert _realign(sd, src=K(D=12)) == 2                         # D*2 not a multiple of 16
    assert _realign(sd, src=K(D=0)) == 1
    assert _realign(sd, src=K(data=A + 8)) == 2                  # not 16-byte aligned
    assert _realign(sd, src=K(data=None)) == 1
    assert _realign(sd, src=K(cap=9)) == 1                       # src cap < W_in
    assert _realign(sd, dst=K(data=A + (1 << 30), cap=9)) == 1   # dst cap < W_in
    assert _realign(sd, dst=K(data=A + (1 << 30), H=3)) == 1     # shapes differ
    assert _realign(sd, dst=K(data=A + 4096)) == 1               # partial overlap
    assert _realign(sd, dst=K(data=A, cap=65)) == 1              # same base, different cap
    assert _realign(sd, k=-1) == 1
    assert _realign(sd, W_in=3) == 1
    assert _realign(sd, pad_in=None) == 1
    assert _realign(sd, w_new=A + 2) == 2


def test_realign_empty_cache_is_a_noop(sd):
    _no_gpu()
    assert _realign(sd, src=_kv(sd, L=0), dst=_kv(sd, data=A + (1 << 30), L=0)) == 0


def test_posmask_rejects(sd):
    _no_gpu()
    f = sd.lib.specdec_build_posmask
    assert f(PO, WN, 2, 3, POS, MSK, 3, None, None) == 1         # pm_cap < k+1
    assert f(None, WN, 2, 3, POS, MSK, 64, None, None) == 1
    assert f(PO, WN, 2, 3, POS + 4, MSK, 64, None, None) == 2    # pos not 8-byte aligned
    assert f(PO, WN, -1, 3, POS, MSK, 64, None, None) == 1
    assert f(PO, WN, 2, 3, POS, POS + 1000, 64, None, None) == 1  # mask inside pos
    assert f(PO, WN, 2, 3, PO - 8, MSK, 64, None, None) == 1     # pos over pad_out
    assert f(None, None, 0, 3, None, None, 64, None, None) == 0   # empty batch


def test_step_rejects(sd):
    _no_gpu()
    src, dst = _kv(sd), _kv(sd, data=A + (1 << 30))
    ws = sd.workspace_bytes(2, 3, 100)
    S_IN, S_OUT = A + (2 << 30), A + (3 << 30)

    def step(B=2, pm_cap=64, src=src, dst=dst, ws_bytes=ws, s_in=None, s_in_stride=0, s_out=None, s_out_stride=0,
             pad_out=PO, pos=POS):
        return sd.lib.specdec_step(LG, 1, DR, PI, B, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst), TK, NA, BO,
                                   pad_out, WN, pos, MSK, pm_cap, s_in, s_in_stride, s_out, s_out_stride, -1, WS,
                                   ws_bytes, None, None, None)
    assert step(pm_cap=13) == 1                  # pm_cap < W_in + k + 1
    assert step(src=_kv(sd, B=3), dst=_kv(sd, data=A + (1 << 30), B=3)) == 1   # cache rows differ
    assert step(ws_bytes=8) == 4
    # token row: short strides, a missing half, overlap, in place with unequal strides
    assert step(s_in=S_IN, s_in_stride=6, s_out=S_OUT, s_out_stride=11) == 1    # s_in_stride < W_in - k
    assert step(s_in=S_IN, s_in_stride=7, s_out=S_OUT, s_out_stride=10) == 1    # s_out_stride < W_in + 1
    assert step(s_in=S_IN, s_in_stride=7, s_out=None, s_out_stride=11) == 1
    assert step(s_in=S_IN, s_in_stride=16, s_out=S_IN + 16, s_out_stride=16) == 1
    assert step(s_in=S_IN, s_in_stride=12, s_out=S_IN, s_out_stride=16) == 1
    assert step(s_in=S_IN + 2, s_in_stride=16, s_out=S_OUT, s_out_stride=16) == 2   # misaligned
    assert step(pad_out=PI) == 1                 # pad_out aliasing pad_in
    assert step(pos=NA - 8) == 1                 # pos over n_acc


def test_bound_call_passes_its_stored_arguments(sd):
    """specdec.Bound converts each argument once to the type the function
    declares and passes the stored values on every call: a step that fails
    validation (pm_cap below W_in + k + 1) fails the same way on each call."""
    _no_gpu()
    src, dst = _kv(sd), _kv(sd, data=A + (1 << 30))
    args = (LG, 1, DR, PI, 2, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst), TK, NA, BO, PO, WN, POS, MSK, 13,
            None, 0, None, 0, -1, WS, sd.workspace_bytes(2, 3, 100), None, None, None)
    call = sd.Bound(sd.lib.specdec_step, args, (src, dst))
    for _ in range(2):
        with pytest.raises(sd.SpecdecError) as e:
            call()
        assert e.value.code == 1 and "pm_cap=13 < W_in+k+1=14" in str(e.value)


def test_bind_step_checks_its_arguments_once(sd):
    """bind_step runs the wrapper's checks when it binds: host tensors and a
    workspace handed to the no-allocation step are refused there."""
    import torch
    B, k, V, W_in = 2, 3, 100, 10
    lg = torch.zeros(B, k + 1, V)
    i32 = lambda *shape: torch.zeros(*shape, dtype=torch.int32)   # noqa: E731
    kv = torch.zeros(1, 2, B, 1, 16, 8, dtype=torch.bfloat16)
    args = (lg, i32(B, k), i32(B), W_in, kv, kv, i32(B, k + 1), i32(B), i32(B), i32(B), i32(1),
            torch.zeros(B, 16, dtype=torch.int64), torch.zeros(B, 16, dtype=torch.uint8))
    with pytest.raises(ValueError, match="contiguous device tensor"):
        sd.bind_step(*args, torch.zeros(64, dtype=torch.int64))
    with pytest.raises(ValueError, match="takes no workspace"):
        sd.bind_step(*args, torch.zeros(64, dtype=torch.int64), noalloc=True)


def test_step_noalloc_rejects_beyond_its_scratch(sd):
    """specdec_step_noalloc refuses, before any HIP call, a step whose
    verification needs more than the library's scratch, and names the limit."""
    _no_gpu()
    limit = int(re.search(r"#define SPECDEC_NOALLOC_SCRATCH_BYTES (\d+)", HEADER).group(1))
    src, dst = _kv(sd, B=16384), _kv(sd, data=A + (1 << 30), B=16384)
    B, k, V = 16384, 7, 128256
    assert sd.workspace_bytes(B, k, V) > limit
    r = sd.lib.specdec_step_noalloc(LG, 1, DR, PI, B, k, V, 16, ctypes.byref(src), ctypes.byref(dst), TK, NA, BO,
                                    PO, WN, POS, MSK, 64, None, 0, None, 0, -1, None, None, None)
    assert r == sd.ERR_WORKSPACE
    msg = sd.lib.specdec_last_error().decode()
    assert str(limit) in msg and "specdec_step_noalloc" in msg
    # an empty batch needs no scratch and returns before any device call
    src, dst = _kv(sd, B=0), _kv(sd, data=A + (1 << 30), B=0)
    assert sd.lib.specdec_step_noalloc(None, 1, None, None, 0, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst),
                                       None, None, None, None, None, None, None, 64, None, 0, None, 0, -1, None,
                                       None, None) == 0


def test_realign_tokens_rejects(sd):
    _no_gpu()
    f = sd.lib.specdec_realign_tokens
    S_IN, S_OUT = A + (2 << 30), A + (3 << 30)
    ok_args = dict(s_in=S_IN, s_in_stride=7, s_out=S_OUT, s_out_stride=11, tokens=A, pad_in=A, n_acc=A, w_new=A,
                   B=2, k=3, W_in=10, pad_id=-1, status=None, stream=None)

    def call(**over):
        d = dict(ok_args)
        d.update(over)
        return f(*d.values())
    assert call(B=-1) == 1
    assert call(k=65) == 1
    assert call(W_in=3) == 1
    assert call(s_in_stride=6) == 1
    assert call(s_out_stride=10) == 1
    assert call(s_out=None) == 1
    assert call(tokens=None) == 1
    assert call(w_new=A + 2) == 2
    assert call(s_out=S_IN, s_out_stride=7) == 1     # in place needs s_out_stride >= W_in + 1 too
    assert call(B=0, s_in=None, s_out=None, tokens=None) == 0


def test_timing_query_rejects_unknown_kernel(sd):
    assert sd.lib.specdec_timing_query(9, None, None) == 1
    assert sd.lib.specdec_timing_query(-1, None, None) == 1
    assert sd.lib.specdec_timing_enable(0) == 0
    assert sd.lib.specdec_timing_enable(511) == 0
    assert sd.lib.specdec_timing_enable(512) == 1
    assert sd.lib.specdec_timing_enable(0) == 0
    assert sd.lib.specdec_timing_enable(-1) == 1


def test_workspace_init_argument_checks(sd):
    _no_gpu()
    assert sd.lib.specdec_workspace_init(None, 0, None) == 0
    assert sd.lib.specdec_workspace_init(None, 16, None) == 4


POOL = A + (4 << 30)
BTOK, PTOK = A + (5 << 30), A + (6 << 30)


def _gather(sd, pool=None, batch=None, **over):
    pool = pool if pool is not None else _kv(sd, data=POOL, B=5, cap=64)
    batch = batch if batch is not None else _kv(sd, B=2, cap=32)
    args = dict(pool_tok=PTOK, pool_tok_stride=65, lens=NA, slots=DR, B=2, Lb=20, k=3, batch_tok=BTOK,
                btok_stride=21, pad_id=-1, pads=PO, pos=POS, mask=MSK, pm_cap=24, status=None, stream=None)
    args.update(over)
    a = list(args.values())
    return sd.lib.specdec_gather_batch(ctypes.byref(pool), *a[:7], ctypes.byref(batch), *a[7:])


def test_gather_rejects(sd):
    _no_gpu()
    K = lambda **kw: _kv(sd, **kw)
    assert _gather(sd, Lb=-1) == 1
    assert _gather(sd, Lb=33) == 1                                   # batch cap < Lb
    assert _gather(sd, B=3) == 1                                     # batch rows differ
    assert _gather(sd, batch=K(B=2, cap=32, H=3)) == 1               # shapes differ
    assert _gather(sd, pool=K(data=A + 4096, B=5, cap=64)) == 1      # pool overlaps the batch
    assert _gather(sd, pool=K(data=POOL, B=0, cap=64)) == 1          # no slot
    assert _gather(sd, lens=None) == 1
    assert _gather(sd, slots=DR + 2) == 2
    assert _gather(sd, pads=None) == 1
    assert _gather(sd, btok_stride=20) == 1                          # < Lb + 1
    assert _gather(sd, pool_tok=None) == 1                           # batch_tok without pool_tok
    assert _gather(sd, pool_tok_stride=0) == 1
    assert _gather(sd, batch_tok=PTOK + 64) == 1                     # token rows overlap
    assert _gather(sd, pm_cap=23) == 1                               # < Lb + k + 1
    assert _gather(sd, mask=None) == 1                               # pos without mask
    assert _gather(sd, pos=POS + 4) == 2
    assert _gather(sd, pads=NA + 4) == 1                             # pads over the lengths
    assert _gather(sd, mask=POS + 64) == 1                           # mask inside pos
    assert _gather(sd, pos=POOL) == 1                                # pos over the pool cache
    assert _gather(sd, k=65) == 1
    assert _gather(sd, batch=K(B=2, cap=32, D=12)) == 2
    assert _gather(sd, B=0, batch=K(B=0, cap=32), lens=None, slots=None, pads=None) == 0   # empty batch


def test_gather_valid_arguments_pass_validation(sd):
    """The same call with valid arguments would be enqueued (only checked with
    an empty batch here, so no kernel is launched)."""
    _no_gpu()
    assert _gather(sd, B=0, batch=_kv(sd, B=0, cap=32)) == 0


def _scatter(sd, pool=None, batch=None, **over):
    pool = pool if pool is not None else _kv(sd, data=POOL, B=5, cap=64)
    batch = batch if batch is not None else _kv(sd, B=2, cap=32)
    args = dict(pads=PO, tokens=TK, n_acc=NA, slots=DR, B=2, k=3, Lb=20)
    rest = dict(pool_tok=PTOK, pool_tok_stride=65, lens=PI, batch_tok=BTOK, btok_stride=25, mode=0, status=None,
                stream=None)
    args.update({k: v for k, v in over.items() if k in args})
    rest.update({k: v for k, v in over.items() if k in rest})
    return sd.lib.specdec_scatter_accepted(ctypes.byref(batch), *args.values(), ctypes.byref(pool), *rest.values())


def test_scatter_rejects(sd):
    _no_gpu()
    K = lambda **kw: _kv(sd, **kw)
    assert _scatter(sd, mode=2) == 1
    assert _scatter(sd, Lb=29) == 1                                  # batch cap < Lb + k + 1
    assert _scatter(sd, k=-1) == 1
    assert _scatter(sd, B=3) == 1
    assert _scatter(sd, pool=K(data=A + 4096, B=5, cap=64)) == 1
    assert _scatter(sd, pads=None) == 1
    assert _scatter(sd, tokens=None) == 1
    assert _scatter(sd, n_acc=NA + 2) == 2
    assert _scatter(sd, lens=NA) == 1                                # lengths over n_acc
    assert _scatter(sd, lens=POOL + 128) == 1                        # lengths inside the pool cache
    assert _scatter(sd, pool_tok=None) == 1
    assert _scatter(sd, pool_tok_stride=0) == 1
    assert _scatter(sd, btok_stride=24) == 1                         # < Lb + k + 2
    assert _scatter(sd, batch_tok=PTOK) == 1                         # token rows overlap
    assert _scatter(sd, lens=None) == 1
    assert _scatter(sd, B=0, batch=K(B=0, cap=32), pads=None, tokens=None, n_acc=None, slots=None,
                    lens=None) == 0


def _sample(sd, **over):
    args = dict(logits=LG, draft_logits=DL, dtype=1, draft=DR, pad_in=PI, u_accept=UA, u_sample=US, T=0.8,
                B=2, k=3, V=100, W_in=10, tokens=TK, n_acc=NA, bonus=BO, pad_out=PO, w_new=WN, ws=WS,
                ws_bytes=sd.sample_workspace_bytes(2, 3, 100), status=None, stream=None)
    args.update(over)
    return sd.lib.specdec_verify_sample(*args.values())


@pytest.mark.parametrize("over,code", [
    (dict(B=-1), 1), (dict(k=65), 1), (dict(V=0), 1), (dict(W_in=3), 1), (dict(dtype=5), 2),
    (dict(T=0.0), 1), (dict(T=-1.0), 1), (dict(T=float("inf")), 1), (dict(T=float("nan")), 1), (dict(T=1e-39), 1),
    (dict(logits=None), 1), (dict(draft_logits=None), 1), (dict(u_accept=None), 1), (dict(u_sample=None), 1),
    (dict(draft=None), 1), (dict(w_new=None), 1), (dict(logits=LG + 1), 2), (dict(u_sample=US + 2), 2),
    (dict(ws=None), 4), (dict(ws=WS + 4), 4), (dict(ws_bytes=64), 4), (dict(B=40000, k=20), 1),
    (dict(pad_out=PI), 1), (dict(tokens=UA), 1), (dict(ws=DL + 128), 1),
])
def test_verify_sample_rejects(sd, over, code):
    _no_gpu()
    assert _sample(sd, **over) == code
    assert sd.lib.specdec_last_error().decode() != ""


def test_verify_sample_empty_and_workspace(sd):
    _no_gpu()
    assert _sample(sd, B=0, logits=None, draft_logits=None, draft=None, pad_in=None, u_accept=None, u_sample=None,
                   tokens=None, n_acc=None, pad_out=None, w_new=None, ws=None) == 0
    # k = 0 needs no draft tensors
    assert sd.sample_workspace_bytes(8, 5, 32000) == 256 + 8 * 16 + (8 * 11 + 8 + 8 * 1) * 16 * 8
    assert sd.sample_workspace_bytes(-1, 0, 5) == 0 and sd.sample_workspace_bytes(1, 65, 5) == 0


def test_rollback_rejects(sd):
    _no_gpu()
    f = sd.lib.specdec_rollback
    T, N, PI, NO, BO, PO, W = A, A + 4096, A + 8192, A + 12288, A + 16384, A + 20480, A + 24576
    assert f(T, N, PI, -1, 3, 10, NO, BO, PO, W, None, None) == 1
    assert f(T, N, PI, 2, 65, 100, NO, BO, PO, W, None, None) == 1
    assert f(T, N, PI, 2, 3, 3, NO, BO, PO, W, None, None) == 1          # W_in < k+1
    assert f(T, None, PI, 2, 3, 10, NO, BO, PO, W, None, None) == 1
    assert f(T, N, PI, 2, 3, 10, NO, BO + 2, PO, W, None, None) == 2
    assert f(T, N, PI, 2, 3, 10, NO, N, PO, W, None, None) == 1          # bonus_out over n_acc_in
    assert f(T, N, PI, 2, 3, 10, N + 4, BO, PO, W, None, None) == 1      # partial overlap, not in place
    assert f(T, N, PI, 2, 3, 10, NO, BO, T + 8, W, None, None) == 1      # pad_out over tokens
    assert f(None, None, None, 0, 3, 10, None, None, None, None, None, None) == 0


def _vdesc(sd, data=A, L=2, H=2, D=8, T=100):
    return sd.Varlen(data, L, H, D, T)


def test_varlen_rollback_rejects(sd):
    _no_gpu()
    f = sd.lib.specdec_varlen_rollback
    S, Dd = _vdesc(sd), _vdesc(sd, data=A + (1 << 30))
    CI, NA, CO, PS = A + (2 << 30), A + (3 << 30), A + (4 << 30), A + (5 << 30)

    def call(src=S, dst=Dd, cu_in=CI, n_acc=NA, B=3, k=2, max_len=20, cu_out=CO, pos=PS, pos_cap=100):
        return f(ctypes.byref(src), ctypes.byref(dst), cu_in, n_acc, B, k, max_len, cu_out, pos, pos_cap, None, None)
    assert f(None, ctypes.byref(Dd), CI, NA, 3, 2, 20, CO, PS, 100, None, None) == 1
    assert call(dst=_vdesc(sd, data=A + (1 << 30), H=3)) == 1              # shapes differ
    assert call(src=_vdesc(sd, D=4, H=1), dst=_vdesc(sd, data=A + (1 << 30), D=4, H=1)) == 2   # H*D not 8k
    assert call(dst=_vdesc(sd, data=A + (1 << 30), T=99)) == 1             # dst smaller
    assert call(max_len=2) == 1                                            # < k+1
    assert call(B=-1) == 1 and call(k=65) == 1
    assert call(cu_out=None) == 1 and call(cu_in=None) == 1
    assert call(pos=PS + 4) == 2
    assert call(pos_cap=99) == 1
    assert call(dst=_vdesc(sd, data=A + 4096)) == 1                        # caches overlap
    assert call(cu_out=CI + 4) == 1                                        # cu_out over cu_in
    assert call(pos=NA) == 1                                               # positions over n_acc
    assert call(pos=A + (1 << 30) + 256) == 1                              # positions inside the dst cache
    assert call(src=_vdesc(sd, data=A + 8), dst=_vdesc(sd, data=A + (1 << 30))) == 2
    assert call(B=0, cu_in=None, n_acc=None, cu_out=None) == 0


def _overlap(sd, rc):
    assert rc == 1 and "overlap" in sd.lib.specdec_last_error().decode(), sd.lib.specdec_last_error().decode()


def test_every_output_stands_apart(sd):
    """Caches, token rows and the status word are outputs like the others: an
    output over any input or over another output is refused before anything
    is enqueued.  (An in-place cache or token row counts once, as an output:
    the GPU tests run those cases.)"""
    _no_gpu()
    CACHE = A + (1 << 30)                    # the dst cache spans 32 KiB from here
    S_IN, S_OUT = A + (2 << 30), A + (3 << 30)
    _overlap(sd, _verify(sd, status=TK))  # status word over tokens
    _overlap(sd, _verify(sd, status=WS + 256))  # status word inside the workspace
    _overlap(sd, _sample(sd, status=US))
    # realignment alone: device values inside the destination, the status word too
    _overlap(sd, _realign(sd, pad_in=CACHE + 64))
    _overlap(sd, _realign(sd, w_new=CACHE + 32764))
    _overlap(sd, _realign(sd, src=_kv(sd, data=CACHE), dst=_kv(sd, data=CACHE), n_acc=CACHE + 4096))  # in place
    f = sd.lib.specdec_realign_kv
    src, dst = _kv(sd), _kv(sd, data=CACHE)
    _overlap(sd, f(ctypes.byref(src), ctypes.byref(dst), 3, 10, PI, NA, WN, CACHE + 16, None))   # status word
    # position ids / mask
    _overlap(sd, sd.lib.specdec_build_posmask(PO, WN, 2, 3, POS, MSK, 64, MSK + 8, None))
    # token row alone
    g = sd.lib.specdec_realign_tokens
    _overlap(sd, g(S_IN, 7, S_OUT, 11, S_OUT + 8, PI, NA, WN, 2, 3, 10, -1, None, None))  # tokens inside s_out
    _overlap(sd, g(S_IN, 7, S_OUT, 11, TK, PI, NA, WN, 2, 3, 10, -1, S_OUT + 4, None))  # status inside s_out
    _overlap(sd, g(S_IN, 16, S_IN, 16, TK, S_IN + 8, NA, WN, 2, 3, 10, -1, None, None))  # in place over pad_in
    # fused steps
    ws = sd.workspace_bytes(2, 3, 100)

    def step(logits=LG, tokens=TK, n_acc=NA, pos=POS, status=None, src=None, dst=None, s_in=None, s_out=None,
             stride=16, pad_in=PI):
        src = src if src is not None else _kv(sd)
        dst = dst if dst is not None else _kv(sd, data=CACHE)
        return sd.lib.specdec_step(logits, 1, DR, pad_in, 2, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst), tokens,
                                   n_acc, BO, PO, WN, pos, MSK, 64, s_in, stride, s_out, stride, -1, WS, ws,
                                   status, None, None)
    _overlap(sd, step(tokens=CACHE + 1024))  # verification output inside the dst cache
    _overlap(sd, step(logits=CACHE))  # logits inside the dst cache
    _overlap(sd, step(status=NA))  # status word over n_acc
    _overlap(sd, step(pos=A + 256))  # positions over the source cache
    _overlap(sd, step(s_in=S_IN, s_out=TK))  # token row over tokens
    _overlap(sd, step(s_in=S_IN, s_out=S_OUT, pos=S_IN + 64))  # positions over the old token row
    _overlap(sd, step(src=_kv(sd, data=CACHE), pad_in=CACHE + 8))  # in place, pad_in inside the cache
    sws = sd.sample_workspace_bytes(2, 3, 100)
    src, dst = _kv(sd), _kv(sd, data=CACHE)
    h = sd.lib.specdec_step_sample
    _overlap(sd, h(LG, DL, 1, DR, PI, UA, CACHE + 512, 0.8, 2, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst), TK, NA, BO,
             PO, WN, POS, MSK, 64, None, 0, None, 0, -1, WS, sws, None, None, None))  # u_sample in the cache
    _overlap(sd, h(LG, DL, 1, DR, PI, UA, US, 0.8, 2, 3, 100, 10, ctypes.byref(src), ctypes.byref(dst), TK, NA, BO,
             PO, WN, POS, MSK, 64, None, 0, None, 0, -1, WS, sws, DL + 4, None, None))  # status word over draft logits
    # Family A rollback: the width and the status word stand apart
    r = sd.lib.specdec_rollback
    T, N, P_, NO, B_, PO_, W = A, A + 4096, A + 8192, A + 12288, A + 16384, A + 20480, A + 24576
    _overlap(sd, r(T, N, P_, 2, 3, 10, NO, B_, PO_, N, None, None))  # w_new over n_acc_in
    _overlap(sd, r(T, N, P_, 2, 3, 10, NO, B_, PO_, W, NO + 4, None))  # status word over n_acc_out


def test_missing_library_fails_loudly(tmp_path):
    """With no built library the binding refuses to import (no fallback path),
    and so do the smoke check and the benchmark, which go through it."""
    import os
    import subprocess
    import sys
    env = dict(os.environ, SPECDEC_LIB=str(tmp_path / "libspecdec.so"))
    for code in ("from paper_2510_22876_amd import specdec",
                 "import __graft_entry__ as g; g.smoke()"):
        r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                           timeout=300)
        assert r.returncode != 0, code
        assert "is not built" in r.stderr, r.stderr[-2000:]
