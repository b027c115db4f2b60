"""Oracle for the greedy verify + KV realign step (EqSpec, arXiv 2510.22876).

TEST INFRASTRUCTURE ONLY.  A plain, slow, scalar CPU implementation (C in
``specdec_oracle.c``, compiled with gcc, called through ctypes on numpy
arrays) that the HIP library is checked against.  It shares no code with the
library and is never imported by the product path; only ``tests/``, the smoke
check and the CPU-baseline leg of the benchmark use it.

Each function names the passage of the paper it follows; the C source header
lists the readings taken where the paper is silent.  Every function here is
pinned by the ``-m "not gpu"`` tests (brute force, closed forms, the paper's
corollaries and invariants, an independent replay of each row alone).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "specdec_oracle.c"
_LIB_PATH = _HERE / "libspecdec_oracle.so"

F32, BF16, F16 = 0, 1, 2
DTYPE_CODE = {"f32": F32, "bf16": BF16, "f16": F16}


def build(force: bool = True) -> Path:
    """Compile the oracle with gcc (plain -O2, no vector intrinsics)."""
    if force or not _LIB_PATH.exists():
        tmp = _LIB_PATH.with_suffix(".so.tmp")
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                        str(_SRC), "-o", str(tmp), "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class Oracle:
    """ctypes handle on one build of the oracle library (tests load mutant builds too)."""

    def __init__(self, path: Path | str | None = None):
        if path is None and os.environ.get("SPECDEC_ORACLE_LIB"):
            path = os.environ["SPECDEC_ORACLE_LIB"]      # another build, e.g. with sanitizers
        if path is None:
            if not _LIB_PATH.exists():
                build(force=False)
            path = _LIB_PATH
        lib = ctypes.CDLL(str(path))
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        lib.oracle_argmax.argtypes = [P, ctypes.c_int, i64]
        lib.oracle_argmax.restype = i64
        lib.oracle_verify.argtypes = [P, ctypes.c_int, P, P, i32, i32, i64, i32, P, P, P, P, P]
        lib.oracle_verify.restype = ctypes.c_int
        lib.oracle_realign_kv.argtypes = [P, i64, P, i64, i32, i32, i32, i32, i32, i32, P, P, i32]
        lib.oracle_realign_kv.restype = ctypes.c_int
        lib.oracle_posmask.argtypes = [P, i32, i32, i32, P, P, i64]
        lib.oracle_posmask.restype = ctypes.c_int
        lib.oracle_realign_tokens.argtypes = [P, i64, P, i64, P, P, P, i32, i32, i32, i32, i32]
        lib.oracle_realign_tokens.restype = ctypes.c_int
        lib.oracle_gather_batch.argtypes = [P, i64, i32, P, i64, P, P, i32, i32, i32, i32, i32, P, i64, P, i64,
                                            i32, P]
        lib.oracle_gather_batch.restype = ctypes.c_int
        lib.oracle_scatter_accepted.argtypes = [P, i64, i32, P, P, i32, P, P, i32, i32, i32, i32, P, i64, i32, P,
                                                i64, P, P, i64]
        lib.oracle_scatter_accepted.restype = ctypes.c_int
        lib.oracle_verify_sample.argtypes = [P, P, ctypes.c_int, P, P, P, P, ctypes.c_double, i32, i32, i64, i32,
                                             P, P, P, P, P]
        lib.oracle_verify_sample.restype = ctypes.c_int
        lib.oracle_rollback.argtypes = [P, P, P, i32, i32, i32, P, P, P, P]
        lib.oracle_rollback.restype = ctypes.c_int
        lib.oracle_varlen_rollback.argtypes = [P, P, i64, i32, i32, i32, P, P, i32, i32, P, P]
        lib.oracle_varlen_rollback.restype = ctypes.c_int
        self.lib = lib


_default: Oracle | None = None


def _load(o: "Oracle | None" = None):
    global _default
    if o is not None:
        return o.lib
    if _default is None:
        _default = Oracle()
    return _default.lib


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _raw_logits(logits, dtype: str):
    """Accept numpy arrays (uint16 bit patterns for bf16/f16) or CPU torch tensors."""
    try:
        import torch
        if isinstance(logits, torch.Tensor):
            t = logits.detach().cpu().contiguous()
            if t.dtype in (torch.bfloat16, torch.float16):
                return t.view(torch.int16).numpy().view(np.uint16)
            return t.numpy()
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(logits)
    if dtype == "f32":
        return _c(a, np.float32)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    return _c(a, np.uint16)


def argmax(row, dtype: str = "f32", oracle: Oracle | None = None) -> int:
    """Greedy prediction of one logit row (Algorithm 3, argmax over the vocabulary):
    lowest index of the maximum, first NaN wins."""
    r = _raw_logits(row, dtype).reshape(-1)
    return int(_load(oracle).oracle_argmax(_ptr(r), DTYPE_CODE[dtype], r.size))


def verify(logits, dtype: str, draft, pad_in, W_in: int, oracle: Oracle | None = None):
    """BatchVerify (Algorithm 3) plus the new width and offsets (Eq. 1 and Eq. 2).

    logits [B][k+1][V]; draft [B][k]; pad_in [B].  Returns a dict with
    tokens [B][k+1], n_acc [B], bonus [B], pad_out [B], w_new (int).
    """
    lg = _raw_logits(logits, dtype)
    B, kp1, V = lg.shape
    k = kp1 - 1
    d = _c(np.asarray(draft).reshape(B, k), np.int32)
    p = _c(np.asarray(pad_in).reshape(B), np.int32)
    tokens = np.zeros((B, k + 1), np.int32)
    n_acc = np.zeros(B, np.int32)
    bonus = np.zeros(B, np.int32)
    pad_out = np.zeros(B, np.int32)
    w_new = np.zeros(1, np.int32)
    rc = _load(oracle).oracle_verify(_ptr(lg), DTYPE_CODE[dtype], _ptr(d), _ptr(p), B, k, V, W_in,
                               _ptr(tokens), _ptr(n_acc), _ptr(bonus), _ptr(pad_out), _ptr(w_new))
    if rc:
        raise OracleError(f"oracle_verify rejected its arguments (code {rc})")
    return dict(tokens=tokens, n_acc=n_acc, bonus=bonus, pad_out=pad_out, w_new=int(w_new[0]))


def verify_sample(logits, draft_logits, dtype: str, draft, pad_in, u_accept, u_sample, temperature: float,
                  W_in: int, oracle: Oracle | None = None):
    """Stochastic (T > 0) verification by speculative sampling: accept draft
    x_r iff u_accept[i][r] * q_r(x_r) < p_r(x_r); at the first rejection the
    correction is drawn from max(0, p_r - q_r) by inversion with u_sample[i];
    after k acceptances the bonus is drawn from p_k.  p = softmax(logits / T),
    q = softmax(draft_logits / T), in double.  Returns the same dict as
    ``verify`` (tokens[i][0..n_acc] are the accepted drafts and the sampled
    token, -1 beyond)."""
    lg = _raw_logits(logits, dtype)
    dl = _raw_logits(draft_logits, dtype)
    B, kp1, V = lg.shape
    k = kp1 - 1
    assert dl.shape == (B, k, V)
    dr = _c(np.asarray(draft).reshape(B, k), np.int32)
    pad = _c(np.asarray(pad_in).reshape(B), np.int32)
    ua = _c(np.asarray(u_accept).reshape(B, k), np.float32)
    us = _c(np.asarray(u_sample).reshape(B), np.float32)
    tokens = np.zeros((B, kp1), np.int32)
    n_acc = np.zeros(B, np.int32)
    bonus = np.zeros(B, np.int32)
    pad_out = np.zeros(B, np.int32)
    w_new = np.zeros(1, np.int32)
    rc = _load(oracle).oracle_verify_sample(_ptr(lg), _ptr(dl), DTYPE_CODE[dtype], _ptr(dr), _ptr(pad), _ptr(ua),
                                            _ptr(us), float(temperature), B, k, V, W_in, _ptr(tokens), _ptr(n_acc),
                                            _ptr(bonus), _ptr(pad_out), _ptr(w_new))
    if rc:
        raise OracleError(f"oracle_verify_sample rejected its arguments (code {rc})")
    return dict(tokens=tokens, n_acc=n_acc, bonus=bonus, pad_out=pad_out, w_new=int(w_new[0]))


def rollback(tokens, n_acc, pad_in, W_in: int, oracle: Oracle | None = None):
    """Family A rollback: every row truncated to the batch-minimum accepted
    count m; returns dict(n_acc (all m), bonus = tokens[i][m], pad_out, w_new)
    by Eq. (1) and Eq. (2) with a_i = m + 1."""
    tk = _c(np.asarray(tokens), np.int32)
    B, kp1 = tk.shape
    na = _c(np.asarray(n_acc).reshape(B), np.int32)
    pad = _c(np.asarray(pad_in).reshape(B), np.int32)
    out = dict(n_acc=np.zeros(B, np.int32), bonus=np.zeros(B, np.int32), pad_out=np.zeros(B, np.int32))
    w = np.zeros(1, np.int32)
    rc = _load(oracle).oracle_rollback(_ptr(tk), _ptr(na), _ptr(pad), B, kp1 - 1, W_in, _ptr(out["n_acc"]),
                                       _ptr(out["bonus"]), _ptr(out["pad_out"]), _ptr(w))
    if rc:
        raise OracleError(f"oracle_rollback rejected its arguments (code {rc})")
    out["w_new"] = int(w[0])
    return out


def varlen_rollback(src, cu_in, n_acc, k: int, dst=None, oracle: Oracle | None = None):
    """Family B rollback on a flat cache [L][2][T_cap][H][D] (uint16 bf16
    bits): sequence i keeps its first len_i - (k - n_acc[i]) rows, compacted;
    returns (dst, cu_out int32 [B+1], pos int64 [T_cap] (rows beyond cu_out[B]
    are -1))."""
    sb = _kv_bits(src) if not isinstance(src, np.ndarray) else _c(src, np.uint16)
    nl, two, T_cap, H, D = sb.shape
    cu = _c(np.asarray(cu_in).reshape(-1), np.int32)
    B = cu.size - 1
    na = _c(np.asarray(n_acc).reshape(B), np.int32)
    out = np.zeros_like(sb) if dst is None else dst
    cu_out = np.zeros(B + 1, np.int32)
    pos = np.full(T_cap, -1, np.int64)
    rc = _load(oracle).oracle_varlen_rollback(_ptr(sb), _ptr(out), T_cap, nl, H, D, _ptr(cu), _ptr(na), B, k,
                                              _ptr(cu_out), _ptr(pos))
    if rc:
        raise OracleError(f"oracle_varlen_rollback rejected its arguments (code {rc})")
    return out, cu_out, pos


def _kv_bits(kv):
    try:
        import torch
        if isinstance(kv, torch.Tensor):
            return kv.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    except ImportError:  # pragma: no cover
        pass
    return _c(kv, np.uint16)


def realign_kv(src, k: int, W_in: int, pad_in, n_acc, w_new: int, dst=None, dst_cap=None,
               oracle: Oracle | None = None):
    """Unpad-append-repad of the KV cache (Section 3.1; Theorem B.1's relocation).

    src: bf16 [n_layers][2][B][H][cap][D] as uint16 bit patterns (or a torch
    bf16 tensor).  Returns dst (uint16, same layout, ``dst_cap`` columns);
    columns [0, w_new) are the result.  When ``dst`` is given it is written in
    place of a fresh array (columns beyond w_new keep their contents).
    """
    s = _kv_bits(src)
    nl, two, B, H, cap, D = s.shape
    assert two == 2
    if dst is None:
        dcap = dst_cap if dst_cap is not None else cap
        dst = np.zeros((nl, 2, B, H, dcap, D), np.uint16)
    assert dst.dtype == np.uint16 and dst.flags["C_CONTIGUOUS"]
    p = _c(np.asarray(pad_in).reshape(B), np.int32)
    a = _c(np.asarray(n_acc).reshape(B), np.int32)
    rc = _load(oracle).oracle_realign_kv(_ptr(s), cap, _ptr(dst), dst.shape[4], nl, B, H, D, k, W_in,
                                   _ptr(p), _ptr(a), int(w_new))
    if rc:
        raise OracleError(f"oracle_realign_kv rejected its arguments (code {rc})")
    return dst


def posmask(pad_out, w_new: int, k: int, pm_cap: int | None = None, oracle: Oracle | None = None):
    """Position ids and attention mask of invariant I2, columns [0, w_new+k+1).

    Returns (pos int64 [B][pm_cap], mask uint8 [B][pm_cap]); columns beyond
    w_new+k+1 are zero.
    """
    p = _c(np.asarray(pad_out).reshape(-1), np.int32)
    B = p.size
    cap = pm_cap if pm_cap is not None else w_new + k + 1
    pos = np.zeros((B, cap), np.int64)
    mask = np.zeros((B, cap), np.uint8)
    rc = _load(oracle).oracle_posmask(_ptr(p), int(w_new), B, k, _ptr(pos), _ptr(mask), cap)
    if rc:
        raise OracleError(f"oracle_posmask rejected its arguments (code {rc})")
    return pos, mask


def realign_tokens(s_in, tokens, pad_in, n_acc, w_new: int, W_in: int, pad_id: int, out_stride=None,
                   oracle: Oracle | None = None):
    """Token row realignment of Alg. 1's phase 3: S[i] <- S[i] + A[i] + B[i], then
    repadding to width L'+1.  s_in int32 [B][>= L+1]; returns int32
    [B][out_stride or L'+1] (columns beyond L'+1 are zero)."""
    si = _c(np.asarray(s_in), np.int32)
    B = si.shape[0]
    tk = _c(np.asarray(tokens), np.int32)
    k = tk.shape[1] - 1
    stride = out_stride if out_stride is not None else w_new + 1
    out = np.zeros((B, stride), np.int32)
    p = _c(np.asarray(pad_in).reshape(B), np.int32)
    a = _c(np.asarray(n_acc).reshape(B), np.int32)
    rc = _load(oracle).oracle_realign_tokens(_ptr(si), si.shape[1], _ptr(out), stride, _ptr(tk), _ptr(p), _ptr(a),
                                             int(w_new), B, k, W_in, int(pad_id))
    if rc:
        raise OracleError(f"oracle_realign_tokens rejected its arguments (code {rc})")
    return out


def gather_batch(pool, pool_tok, lens, slots, Lb: int, batch_cap: int, btok_stride: int, pad_id: int, out=None,
                 oracle: Oracle | None = None):
    """EXSpec's GetBatch (Alg. 2): rows gathered from pool slots and left-padded
    to width Lb.  pool uint16 [L][2][N][H][cap][D]; pool_tok int32 [N][*];
    returns (batch uint16 [L][2][B][H][batch_cap][D], batch_tok int32
    [B][btok_stride], pads int32 [B]).  ``out`` = (batch, batch_tok) writes into
    given arrays (cache columns >= Lb and token columns > Lb keep their
    contents); fresh arrays are zero there."""
    pl = _kv_bits(pool)
    nl, two, N, H, cap, D = pl.shape
    pt = _c(np.asarray(pool_tok), np.int32)
    ln = _c(np.asarray(lens).reshape(N), np.int32)
    sl = _c(np.asarray(slots).reshape(-1), np.int32)
    B = sl.size
    if out is None:
        batch = np.zeros((nl, 2, B, H, batch_cap, D), np.uint16)
        btok = np.zeros((B, btok_stride), np.int32)
    else:
        batch, btok = out
        assert batch.dtype == np.uint16 and batch.flags["C_CONTIGUOUS"] and batch.shape == (nl, 2, B, H, batch_cap, D)
        assert btok.dtype == np.int32 and btok.flags["C_CONTIGUOUS"] and btok.shape == (B, btok_stride)
    pads = np.zeros(B, np.int32)
    rc = _load(oracle).oracle_gather_batch(_ptr(pl), cap, N, _ptr(pt), pt.shape[1], _ptr(ln), _ptr(sl), B, int(Lb),
                                           nl, H, D, _ptr(batch), batch_cap, _ptr(btok), btok_stride, int(pad_id),
                                           _ptr(pads))
    if rc:
        raise OracleError(f"oracle_gather_batch rejected its arguments (code {rc})")
    return batch, btok, pads


def scatter_accepted(batch, pads, tokens, n_acc, slots, Lb: int, pool, pool_tok, lens, batch_tok=None,
                     oracle: Oracle | None = None):
    """EXSpec's write-back (Alg. 2, Phase 4), in place on pool (uint16), pool_tok
    and lens (int32 numpy arrays) and, when given, the batch token row
    batch_tok (int32 [B][stride], the step's append)."""
    bt = _kv_bits(batch)
    nl, two, B, H, bcap, D = bt.shape
    assert pool.dtype == np.uint16 and pool.flags["C_CONTIGUOUS"]
    assert pool_tok.dtype == np.int32 and pool_tok.flags["C_CONTIGUOUS"] and lens.dtype == np.int32
    tk = _c(np.asarray(tokens), np.int32)
    k = tk.shape[1] - 1
    pd = _c(np.asarray(pads).reshape(B), np.int32)
    na = _c(np.asarray(n_acc).reshape(B), np.int32)
    sl = _c(np.asarray(slots).reshape(B), np.int32)
    N, cap = pool.shape[2], pool.shape[4]
    if batch_tok is not None:
        assert batch_tok.dtype == np.int32 and batch_tok.flags["C_CONTIGUOUS"]
        bptr, bstride = _ptr(batch_tok), batch_tok.shape[1]
    else:
        bptr, bstride = None, 0
    rc = _load(oracle).oracle_scatter_accepted(_ptr(bt), bcap, B, _ptr(pd), _ptr(tk), k, _ptr(na), _ptr(sl), int(Lb),
                                               nl, H, D, _ptr(pool), cap, N, _ptr(pool_tok), pool_tok.shape[1],
                                               _ptr(lens), bptr, bstride)
    if rc:
        raise OracleError(f"oracle_scatter_accepted rejected its arguments (code {rc})")


def step(logits, dtype: str, draft, pad_in, kv, W_in: int, dst_cap=None,
         oracle: Oracle | None = None):
    """One whole step: verify, then realign, then position ids and mask."""
    v = verify(logits, dtype, draft, pad_in, W_in, oracle=oracle)
    k = np.asarray(draft).shape[-1]
    out = realign_kv(kv, k, W_in, pad_in, v["n_acc"], v["w_new"], dst_cap=dst_cap, oracle=oracle)
    pos, mask = posmask(v["pad_out"], v["w_new"], k, oracle=oracle)
    v.update(kv=out, pos=pos, mask=mask)
    return v
