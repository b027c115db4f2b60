"""ctypes binding of libspecdec.so (C ABI in include/specdec.h).

Argument marshalling only: torch tensors are passed as device pointers, the
stream is torch's current HIP stream, and every step of the path runs in the
library's HIP kernels.  Importing this module loads the library and raises if
it has not been built; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from pathlib import Path

import torch

# SPECDEC_LIB selects another build of the library (for instance one with a
# host-side sanitizer); the default is the in-tree build.
_LIB_PATH = Path(os.environ.get("SPECDEC_LIB") or Path(__file__).resolve().parent / "libspecdec.so")

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_HIP, ERR_WORKSPACE = 0, 1, 2, 3, 4
F32, BF16, F16 = 0, 1, 2
DTYPE_OF = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}
KERNEL_VERIFY, KERNEL_REALIGN, KERNEL_POSMASK, KERNEL_GATHER, KERNEL_WRITEBACK, KERNEL_SAMPLE = 0, 1, 2, 3, 4, 5
KERNEL_VARLEN, KERNEL_VERIFY_SCAN, KERNEL_SAMPLE_STATS = 6, 7, 8
TIMING_ALL = 511
DEV_BAD_PAD_IN, DEV_BAD_ACCEPT, DEV_BAD_WIDTH, DEV_BAD_PAD_OUT = 1, 2, 4, 8
DEV_BAD_SLOT, DEV_SLOT_LEN, DEV_BAD_UNIFORM = 0x10, 0x20, 0x40
WRITEBACK_FULL, WRITEBACK_APPEND = 0, 1

EXPORTED = (
    "specdec_abi_version", "specdec_last_error", "specdec_workspace_bytes", "specdec_workspace_init",
    "specdec_verify_greedy", "specdec_sample_workspace_bytes", "specdec_verify_sample", "specdec_realign_kv", "specdec_build_posmask", "specdec_realign_tokens",
    "specdec_step", "specdec_step_noalloc", "specdec_step_sample", "specdec_gather_batch", "specdec_scatter_accepted",
    "specdec_rollback", "specdec_varlen_rollback",
    "specdec_sched_create", "specdec_sched_destroy", "specdec_sched_next_batch", "specdec_sched_commit",
    "specdec_sched_lengths", "specdec_sched_active",
    "specdec_timing_enable", "specdec_timing_reset", "specdec_timing_query",
)


class SpecdecError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"specdec error {code}: {msg}")
        self.code = code


class KV(ctypes.Structure):
    """specdec_kv_t: bf16 cache [L][2][B][H][cap][D]."""
    _fields_ = [("data", ctypes.c_void_p), ("L", ctypes.c_int32), ("B", ctypes.c_int32),
                ("H", ctypes.c_int32), ("D", ctypes.c_int32), ("cap", ctypes.c_int64)]


class Varlen(ctypes.Structure):
    """specdec_varlen_t: flat bf16 cache [L][2][T_cap][H][D]."""
    _fields_ = [("data", ctypes.c_void_p), ("L", ctypes.c_int32), ("H", ctypes.c_int32), ("D", ctypes.c_int32),
                ("T_cap", ctypes.c_int64)]


class BatchInfo(ctypes.Structure):
    """specdec_batch_info_t."""
    _fields_ = [("B", ctypes.c_int32), ("width", ctypes.c_int32), ("same_length", ctypes.c_int32),
                ("reuse", ctypes.c_int32)]


def _load(path: Path = _LIB_PATH) -> ctypes.CDLL:
    if not Path(path).exists():
        raise ImportError(f"{path} is not built; run `python -m paper_2510_22876_amd.build`")
    lib = ctypes.CDLL(str(path))
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    pKV = ctypes.POINTER(KV)
    lib.specdec_abi_version.restype = i32
    lib.specdec_last_error.restype = ctypes.c_char_p
    lib.specdec_workspace_bytes.argtypes = [i32, i32, i32]
    lib.specdec_workspace_bytes.restype = sz
    lib.specdec_workspace_init.argtypes = [P, sz, P]
    lib.specdec_verify_greedy.argtypes = [P, i32, P, P, i32, i32, i32, i32, P, P, P, P, P, P, sz, P, P]
    lib.specdec_realign_kv.argtypes = [pKV, pKV, i32, i32, P, P, P, P, P]
    lib.specdec_build_posmask.argtypes = [P, P, i32, i32, P, P, i64, P, P]
    lib.specdec_realign_tokens.argtypes = [P, i64, P, i64, P, P, P, P, i32, i32, i32, i32, P, P]
    lib.specdec_step.argtypes = [P, i32, P, P, i32, i32, i32, i32, pKV, pKV, P, P, P, P, P, P, P, i64,
                                 P, i64, P, i64, i32, P, sz, P, P, P]
    lib.specdec_step_noalloc.argtypes = [P, i32, P, P, i32, i32, i32, i32, pKV, pKV, P, P, P, P, P, P, P, i64,
                                         P, i64, P, i64, i32, P, P, P]
    lib.specdec_sample_workspace_bytes.argtypes = [i32, i32, i32]
    lib.specdec_sample_workspace_bytes.restype = sz
    lib.specdec_verify_sample.argtypes = [P, P, i32, P, P, P, P, ctypes.c_float, i32, i32, i32, i32, P, P, P, P, P,
                                          P, sz, P, P]
    lib.specdec_step_sample.argtypes = [P, P, i32, P, P, P, P, ctypes.c_float, i32, i32, i32, i32, pKV, pKV, P, P, P,
                                        P, P, P, P, i64, P, i64, P, i64, i32, P, sz, P, P, P]
    lib.specdec_rollback.argtypes = [P, P, P, i32, i32, i32, P, P, P, P, P, P]
    pVL = ctypes.POINTER(Varlen)
    lib.specdec_varlen_rollback.argtypes = [pVL, pVL, P, P, i32, i32, i32, P, P, i64, P, P]
    lib.specdec_gather_batch.argtypes = [pKV, P, i64, P, P, i32, i32, i32, pKV, P, i64, i32, P, P, P, i64, P, P]
    lib.specdec_scatter_accepted.argtypes = [pKV, P, P, P, P, i32, i32, i32, pKV, P, i64, P, P, i64, i32, P, P]
    lib.specdec_sched_create.argtypes = [P, i32, i32, i32, i32, i32, i32, ctypes.POINTER(P)]
    lib.specdec_sched_destroy.argtypes = [P]
    lib.specdec_sched_destroy.restype = None
    lib.specdec_sched_next_batch.argtypes = [P, P, P, ctypes.POINTER(BatchInfo)]
    lib.specdec_sched_commit.argtypes = [P, P, P, i32]
    lib.specdec_sched_lengths.argtypes = [P, P]
    lib.specdec_sched_active.argtypes = [P]
    lib.specdec_sched_active.restype = i32
    lib.specdec_timing_enable.argtypes = [i32]
    lib.specdec_timing_query.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    for name in ("specdec_workspace_init", "specdec_verify_greedy", "specdec_realign_kv",
                 "specdec_build_posmask", "specdec_realign_tokens", "specdec_step", "specdec_timing_enable",
                 "specdec_timing_reset", "specdec_timing_query", "specdec_gather_batch",
                 "specdec_scatter_accepted", "specdec_sched_create", "specdec_sched_next_batch", "specdec_verify_sample",
                 "specdec_step_sample", "specdec_rollback", "specdec_varlen_rollback",
                 "specdec_sched_commit", "specdec_sched_lengths"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


lib = _load()
LIB_PATH = str(_LIB_PATH)


def _check(code: int) -> None:
    if code != OK:
        raise SpecdecError(code, lib.specdec_last_error().decode())


def _req(name, t, shape, dtype, optional=False):
    """Marshalling-level check that a tensor matches what the C ABI will assume."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _p(t) -> int | None:
    """Device pointer of a tensor (None for None); raw ints pass through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream or None
    return stream if isinstance(stream, int) else stream.cuda_stream


def kv_desc(t: torch.Tensor) -> KV:
    """Descriptor of a contiguous bf16 cache tensor [L][2][B][H][cap][D]."""
    if t.dim() != 6 or t.shape[1] != 2:
        raise ValueError("KV cache must be [L][2][B][H][cap][D]")
    if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
        raise ValueError("KV cache must be a contiguous bfloat16 device tensor")
    L, _, B, H, cap, D = t.shape
    return KV(t.data_ptr(), L, B, H, D, cap)


def abi_version() -> int:
    return lib.specdec_abi_version()


def workspace_bytes(B: int, k: int, V: int) -> int:
    return lib.specdec_workspace_bytes(B, k, V)


def alloc_workspace(B: int, k: int, V: int, device="cuda") -> torch.Tensor:
    """A workspace tensor for specdec_verify_greedy / specdec_step (needs no
    initialisation)."""
    n = workspace_bytes(B, k, V)
    return torch.empty((n + 7) // 8, dtype=torch.int64, device=device)


def specdec_workspace_init(workspace: torch.Tensor, nbytes: int | None = None, stream=None) -> None:
    n = workspace.numel() * workspace.element_size() if nbytes is None else nbytes
    _check(lib.specdec_workspace_init(_p(workspace), n, _stream(stream)))


def _check_verify(logits, draft, pad_in, tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status):
    if logits.dim() != 3 or logits.dtype not in DTYPE_OF or not logits.is_cuda or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous device tensor [B][k+1][V] of float32/bfloat16/float16")
    B, kp1, V = logits.shape
    i32 = torch.int32
    _req("draft", draft, (B, kp1 - 1), i32)
    _req("pad_in", pad_in, (B,), i32)
    _req("tokens", tokens, (B, kp1), i32)
    _req("n_acc", n_acc, (B,), i32)
    _req("bonus", bonus, (B,), i32, optional=True)
    _req("pad_out", pad_out, (B,), i32)
    _req("w_new", w_new, (1,), i32)
    _req("dev_status", dev_status, (1,), i32, optional=True)
    if workspace is None:   # the library's own scratch (specdec_step_noalloc)
        return
    if workspace.numel() * workspace.element_size() < workspace_bytes(B, kp1 - 1, V) or not workspace.is_cuda:
        raise ValueError("workspace too small")


def specdec_verify_greedy(logits, draft, pad_in, W_in: int, tokens, n_acc, bonus, pad_out, w_new,
                          workspace, dev_status=None, stream=None) -> None:
    B, kp1, V = logits.shape
    _check_verify(logits, draft, pad_in, tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status)
    _check(lib.specdec_verify_greedy(
        _p(logits), DTYPE_OF[logits.dtype], _p(draft), _p(pad_in), B, kp1 - 1, V, W_in,
        _p(tokens), _p(n_acc), _p(bonus), _p(pad_out), _p(w_new),
        _p(workspace), workspace.numel() * workspace.element_size(), _p(dev_status), _stream(stream)))


def sample_workspace_bytes(B: int, k: int, V: int) -> int:
    return lib.specdec_sample_workspace_bytes(B, k, V)


def alloc_sample_workspace(B: int, k: int, V: int, device="cuda") -> torch.Tensor:
    """A workspace tensor for specdec_verify_sample (needs no initialisation)."""
    n = sample_workspace_bytes(B, k, V)
    return torch.empty((n + 7) // 8, dtype=torch.int64, device=device)


def specdec_verify_sample(logits, draft_logits, draft, pad_in, u_accept, u_sample, temperature: float, W_in: int,
                          tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status=None, stream=None) -> None:
    """Stochastic (T > 0) verification by speculative sampling with the
    caller's uniforms (u_accept [B][k], u_sample [B], float32)."""
    if logits.dim() != 3 or logits.dtype not in DTYPE_OF or not logits.is_cuda or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous device tensor [B][k+1][V] of float32/bfloat16/float16")
    B, kp1, V = logits.shape
    k = kp1 - 1
    _req("draft_logits", draft_logits, (B, k, V), logits.dtype)
    _req("draft", draft, (B, k), torch.int32)
    _req("pad_in", pad_in, (B,), torch.int32)
    _req("u_accept", u_accept, (B, k), torch.float32)
    _req("u_sample", u_sample, (B,), torch.float32)
    _req("tokens", tokens, (B, kp1), torch.int32)
    _req("n_acc", n_acc, (B,), torch.int32)
    _req("bonus", bonus, (B,), torch.int32, optional=True)
    _req("pad_out", pad_out, (B,), torch.int32)
    _req("w_new", w_new, (1,), torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    nb = workspace.numel() * workspace.element_size()
    if nb < sample_workspace_bytes(B, k, V) or not workspace.is_cuda:
        raise ValueError("workspace too small")
    _check(lib.specdec_verify_sample(_p(logits), _p(draft_logits), DTYPE_OF[logits.dtype], _p(draft), _p(pad_in),
                                     _p(u_accept), _p(u_sample), float(temperature), B, k, V, W_in, _p(tokens),
                                     _p(n_acc), _p(bonus), _p(pad_out), _p(w_new), _p(workspace), nb,
                                     _p(dev_status), _stream(stream)))


def specdec_realign_kv(src, dst, k: int, W_in: int, pad_in, n_acc, w_new, dev_status=None,
                       stream=None) -> None:
    s = kv_desc(src)
    d = kv_desc(dst)
    _req("pad_in", pad_in, (s.B,), torch.int32)
    _req("n_acc", n_acc, (s.B,), torch.int32)
    _req("w_new", w_new, (1,), torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_realign_kv(ctypes.byref(s), ctypes.byref(d), k, W_in, _p(pad_in), _p(n_acc),
                                  _p(w_new), _p(dev_status), _stream(stream)))


def specdec_build_posmask(pad_out, w_new, k: int, pos, mask, dev_status=None, stream=None) -> None:
    B, pm_cap = pos.shape
    _req("pos", pos, (B, pm_cap), torch.int64)
    _req("mask", mask, (B, pm_cap), torch.uint8)
    _req("pad_out", pad_out, (B,), torch.int32)
    _req("w_new", w_new, (1,), torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_build_posmask(_p(pad_out), _p(w_new), B, k, _p(pos), _p(mask), pm_cap,
                                     _p(dev_status), _stream(stream)))


def specdec_realign_tokens(s_in, s_out, tokens, pad_in, n_acc, w_new, W_in: int, pad_id: int,
                           dev_status=None, stream=None) -> None:
    B, kp1 = tokens.shape
    _req("tokens", tokens, (B, kp1), torch.int32)
    _req("s_in", s_in, (B, s_in.shape[1]), torch.int32)
    _req("s_out", s_out, (B, s_out.shape[1]), torch.int32)
    _req("pad_in", pad_in, (B,), torch.int32)
    _req("n_acc", n_acc, (B,), torch.int32)
    _req("w_new", w_new, (1,), torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_realign_tokens(_p(s_in), s_in.shape[1], _p(s_out), s_out.shape[1], _p(tokens), _p(pad_in),
                                      _p(n_acc), _p(w_new), B, kp1 - 1, W_in, pad_id, _p(dev_status),
                                      _stream(stream)))


def _greedy_step(noalloc, logits, draft, pad_in, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new, pos, mask,
                 workspace, dev_status, sync_w_new, stream, s_in, s_out, pad_id):
    """Checks and marshals the arguments of specdec_step (or, with
    ``noalloc``, specdec_step_noalloc): (function, arguments, host word)."""
    B, kp1, V = logits.shape
    _check_verify(logits, draft, pad_in, tokens, n_acc, bonus, pad_out, w_new, None if noalloc else workspace,
                  dev_status)
    s = kv_desc(src)
    d = kv_desc(dst)
    if s.B != B:
        raise ValueError("cache rows differ from logit rows")
    _req("pos", pos, (B, pos.shape[1]), torch.int64)
    _req("mask", mask, (B, pos.shape[1]), torch.uint8)
    if (s_in is None) != (s_out is None):
        raise ValueError("give both s_in and s_out, or neither")
    if s_in is not None:
        _req("s_in", s_in, (B, s_in.shape[1]), torch.int32)
        _req("s_out", s_out, (B, s_out.shape[1]), torch.int32)
    host = ctypes.c_int32(-1)
    head = (_p(logits), DTYPE_OF[logits.dtype], _p(draft), _p(pad_in), B, kp1 - 1, V, W_in,
            ctypes.byref(s), ctypes.byref(d), _p(tokens), _p(n_acc), _p(bonus), _p(pad_out), _p(w_new),
            _p(pos), _p(mask), pos.shape[1], _p(s_in), s_in.shape[1] if s_in is not None else 0, _p(s_out),
            s_out.shape[1] if s_out is not None else 0, pad_id)
    ws = () if noalloc else (_p(workspace), workspace.numel() * workspace.element_size())
    tail = (_p(dev_status), ctypes.byref(host) if sync_w_new else None, _stream(stream))
    return (lib.specdec_step_noalloc if noalloc else lib.specdec_step), head + ws + tail, host


def specdec_step(logits, draft, pad_in, W_in: int, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                 pos, mask, workspace, dev_status=None, sync_w_new: bool = False, stream=None,
                 s_in=None, s_out=None, pad_id: int = 0):
    """The fused step (with the token row S when ``s_in`` / ``s_out`` are
    given); returns L' as a Python int when ``sync_w_new``."""
    fn, args, host = _greedy_step(False, logits, draft, pad_in, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                                  pos, mask, workspace, dev_status, sync_w_new, stream, s_in, s_out, pad_id)
    _check(fn(*args))
    return host.value if sync_w_new else None


def specdec_step_noalloc(logits, draft, pad_in, W_in: int, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                         pos, mask, dev_status=None, sync_w_new: bool = False, stream=None,
                         s_in=None, s_out=None, pad_id: int = 0):
    """``specdec_step`` on the library's own scratch (no workspace argument);
    returns L' as a Python int when ``sync_w_new``."""
    fn, args, host = _greedy_step(True, logits, draft, pad_in, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                                  pos, mask, None, dev_status, sync_w_new, stream, s_in, s_out, pad_id)
    _check(fn(*args))
    return host.value if sync_w_new else None


class Bound:
    """One library call whose arguments were checked and converted once.

    Each call passes the stored arguments again: the same device buffers (the
    tensors are kept alive here), sizes and stream.  For loops that reuse one
    set of buffers every step, where checking and converting some thirty
    arguments per call costs more host time than the step's kernels take at
    small batches.  New inputs go into the bound tensors in place (``copy_``);
    a tensor that is reallocated or resized needs a new binding."""
    __slots__ = ("_fn", "_args", "_keep")

    def __init__(self, fn, args, keep):
        byref = type(ctypes.byref(ctypes.c_int32()))
        self._args = tuple(a if a is None or isinstance(a, byref) else typ(a) for typ, a in zip(fn.argtypes, args))
        self._fn, self._keep = fn, keep

    def __call__(self) -> None:
        code = self._fn(*self._args)
        if code != OK:
            raise SpecdecError(code, lib.specdec_last_error().decode())


def bind_step(logits, draft, pad_in, W_in: int, src, dst, tokens, n_acc, bonus, pad_out, w_new, pos, mask,
              workspace=None, dev_status=None, stream=None, s_in=None, s_out=None, pad_id: int = 0,
              noalloc: bool = False) -> Bound:
    """``specdec_step`` (``specdec_step_noalloc`` with ``noalloc``, which takes
    no workspace) checked and marshalled once; call the result to run a step.
    The stream is the one given, else the current stream at binding time."""
    if noalloc and workspace is not None:
        raise ValueError("specdec_step_noalloc takes no workspace")
    fn, args, _ = _greedy_step(noalloc, logits, draft, pad_in, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                               pos, mask, workspace, dev_status, False, stream, s_in, s_out, pad_id)
    keep = (logits, draft, pad_in, src, dst, tokens, n_acc, bonus, pad_out, w_new, pos, mask, workspace, dev_status,
            s_in, s_out)
    return Bound(fn, args, keep)


def specdec_gather_batch(pool, pool_tok, lens, slots, Lb: int, batch, pads, batch_tok=None, pos=None, mask=None,
                         k: int = 0, pad_id: int = 0, dev_status=None, stream=None) -> None:
    """EXSpec's GetBatch: rows ``slots`` of the pool gathered into ``batch``,
    left-padded to width ``Lb`` (with token rows, paddings and, when given,
    position ids / mask over [0, Lb + k + 1))."""
    pl = kv_desc(pool)
    bt = kv_desc(batch)
    B = bt.B
    _req("lens", lens, (pl.B,), torch.int32)
    _req("slots", slots, (B,), torch.int32)
    _req("pads", pads, (B,), torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    tok_stride = btok_stride = 0
    if batch_tok is not None:
        _req("pool_tok", pool_tok, (pl.B, pool_tok.shape[1]), torch.int32)
        _req("batch_tok", batch_tok, (B, batch_tok.shape[1]), torch.int32)
        tok_stride, btok_stride = pool_tok.shape[1], batch_tok.shape[1]
    pm_cap = 0
    if pos is not None or mask is not None:
        _req("pos", pos, (B, pos.shape[1]), torch.int64)
        _req("mask", mask, (B, pos.shape[1]), torch.uint8)
        pm_cap = pos.shape[1]
    _check(lib.specdec_gather_batch(ctypes.byref(pl), _p(pool_tok) if batch_tok is not None else None, tok_stride,
                                    _p(lens), _p(slots), B, Lb, k, ctypes.byref(bt), _p(batch_tok), btok_stride,
                                    pad_id, _p(pads), _p(pos), _p(mask), pm_cap, _p(dev_status), _stream(stream)))


def specdec_scatter_accepted(batch, pads, tokens, n_acc, slots, Lb: int, pool, pool_tok, lens, batch_tok=None,
                             mode: int = WRITEBACK_FULL, dev_status=None, stream=None) -> None:
    """EXSpec's write-back: each row's unpadded cache up to its accepted
    entries returns to its pool slot (whole, or only the new entries with
    ``mode=WRITEBACK_APPEND``); the slot's token list and length grow."""
    bt = kv_desc(batch)
    pl = kv_desc(pool)
    B = bt.B
    _req("tokens", tokens, (B, tokens.shape[1]), torch.int32)
    k = tokens.shape[1] - 1
    _req("pads", pads, (B,), torch.int32)
    _req("n_acc", n_acc, (B,), torch.int32)
    _req("slots", slots, (B,), torch.int32)
    _req("lens", lens, (pl.B,), torch.int32)
    _req("pool_tok", pool_tok, (pl.B, pool_tok.shape[1]), torch.int32)
    _req("batch_tok", batch_tok, (B, batch_tok.shape[1] if batch_tok is not None else 0), torch.int32, optional=True)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_scatter_accepted(ctypes.byref(bt), _p(pads), _p(tokens), _p(n_acc), _p(slots), B, k, Lb,
                                        ctypes.byref(pl), _p(pool_tok), pool_tok.shape[1], _p(lens), _p(batch_tok),
                                        batch_tok.shape[1] if batch_tok is not None else 0, mode, _p(dev_status),
                                        _stream(stream)))


class SchedBatch:
    """One batch chosen by the scheduler: its slots (row order), their lengths,
    the width, and whether it is same-length / the previous batch reused."""

    def __init__(self, slots, lens, width, same_length, reuse):
        self.slots, self.lens, self.width = slots, lens, width
        self.same_length, self.reuse = same_length, reuse


class Scheduler:
    """The library's SequencePool scheduler (specdec_sched_*; host only)."""

    def __init__(self, lens, window: int, batch: int, max_new: int, sort_by_length: bool = True,
                 eos_id: int = -1):
        import numpy as np
        ln = np.ascontiguousarray(np.asarray(lens, dtype=np.int32).reshape(-1))
        self._lib = lib
        self._h = ctypes.c_void_p(None)
        self.N = ln.size
        self.batch = batch
        _check(lib.specdec_sched_create(ln.ctypes.data if ln.size else None, ln.size, window, batch, max_new,
                                        1 if sort_by_length else 0, eos_id, ctypes.byref(self._h)))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.specdec_sched_destroy(h)
            self._h = None

    def next_batch(self) -> SchedBatch | None:
        import numpy as np
        slots = np.zeros(max(self.batch, 1), np.int32)
        lens = np.zeros(max(self.batch, 1), np.int32)
        info = BatchInfo()
        _check(lib.specdec_sched_next_batch(self._h, slots.ctypes.data, lens.ctypes.data, ctypes.byref(info)))
        if info.B == 0:
            return None
        return SchedBatch([int(x) for x in slots[:info.B]], [int(x) for x in lens[:info.B]], int(info.width),
                          bool(info.same_length), bool(info.reuse))

    def commit(self, batch: SchedBatch, n_acc, appended) -> None:
        """n_acc[i] accepted drafts; appended[i] the n_acc[i] + 1 tokens row i gained."""
        import numpy as np
        na = np.ascontiguousarray(np.asarray(n_acc, np.int32).reshape(-1))
        k = int(max(len(a) for a in appended)) - 1 if len(appended) else 0
        tok = np.full((max(na.size, 1), k + 1), -1, np.int32)
        for i, a in enumerate(appended):
            tok[i, : len(a)] = a
        _check(lib.specdec_sched_commit(self._h, na.ctypes.data, tok.ctypes.data, k))

    def lengths(self) -> list:
        import numpy as np
        out = np.zeros(max(self.N, 1), np.int32)
        _check(lib.specdec_sched_lengths(self._h, out.ctypes.data))
        return [int(x) for x in out[: self.N]]

    def has_active(self) -> bool:
        return lib.specdec_sched_active(self._h) > 0


def specdec_step_sample(logits, draft_logits, draft, pad_in, u_accept, u_sample, temperature: float, W_in: int,
                        src, dst, tokens, n_acc, bonus, pad_out, w_new, pos, mask, workspace, dev_status=None,
                        sync_w_new: bool = False, stream=None, s_in=None, s_out=None, pad_id: int = 0):
    """The fused step with stochastic verification (speculative sampling with
    the caller's uniforms); returns L' as a Python int when ``sync_w_new``."""
    B, kp1, V = logits.shape
    k = kp1 - 1
    if logits.dtype not in DTYPE_OF or not logits.is_cuda or not logits.is_contiguous():
        raise ValueError("logits must be a contiguous device tensor [B][k+1][V] of float32/bfloat16/float16")
    _req("draft_logits", draft_logits, (B, k, V), logits.dtype)
    for name, t, shape, dt in (("draft", draft, (B, k), torch.int32), ("pad_in", pad_in, (B,), torch.int32),
                               ("u_accept", u_accept, (B, k), torch.float32), ("u_sample", u_sample, (B,), torch.float32),
                               ("tokens", tokens, (B, kp1), torch.int32), ("n_acc", n_acc, (B,), torch.int32),
                               ("pad_out", pad_out, (B,), torch.int32), ("w_new", w_new, (1,), torch.int32)):
        _req(name, t, shape, dt)
    _req("bonus", bonus, (B,), torch.int32, optional=True)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    sdesc, ddesc = kv_desc(src), kv_desc(dst)
    if sdesc.B != B:
        raise ValueError("cache rows differ from logit rows")
    _req("pos", pos, (B, pos.shape[1]), torch.int64)
    _req("mask", mask, (B, pos.shape[1]), torch.uint8)
    if (s_in is None) != (s_out is None):
        raise ValueError("give both s_in and s_out, or neither")
    if s_in is not None:
        _req("s_in", s_in, (B, s_in.shape[1]), torch.int32)
        _req("s_out", s_out, (B, s_out.shape[1]), torch.int32)
    nb = workspace.numel() * workspace.element_size()
    if nb < sample_workspace_bytes(B, k, V) or not workspace.is_cuda:
        raise ValueError("workspace too small")
    host = ctypes.c_int32(-1)
    _check(lib.specdec_step_sample(
        _p(logits), _p(draft_logits), DTYPE_OF[logits.dtype], _p(draft), _p(pad_in), _p(u_accept), _p(u_sample),
        float(temperature), B, k, V, W_in, ctypes.byref(sdesc), ctypes.byref(ddesc), _p(tokens), _p(n_acc), _p(bonus),
        _p(pad_out), _p(w_new), _p(pos), _p(mask), pos.shape[1], _p(s_in), s_in.shape[1] if s_in is not None else 0,
        _p(s_out), s_out.shape[1] if s_out is not None else 0, pad_id, _p(workspace), nb, _p(dev_status),
        ctypes.byref(host) if sync_w_new else None, _stream(stream)))
    return host.value if sync_w_new else None


def specdec_rollback(tokens, n_acc_in, pad_in, W_in: int, n_acc_out, bonus_out, pad_out, w_new, dev_status=None,
                     stream=None) -> None:
    """Family A rollback: every row truncated to the batch-minimum accepted count."""
    B, kp1 = tokens.shape
    for name, t, shape in (("tokens", tokens, (B, kp1)), ("n_acc_in", n_acc_in, (B,)), ("pad_in", pad_in, (B,)),
                           ("n_acc_out", n_acc_out, (B,)), ("bonus_out", bonus_out, (B,)), ("pad_out", pad_out, (B,)),
                           ("w_new", w_new, (1,))):
        _req(name, t, shape, torch.int32)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_rollback(_p(tokens), _p(n_acc_in), _p(pad_in), B, kp1 - 1, W_in, _p(n_acc_out), _p(bonus_out),
                                _p(pad_out), _p(w_new), _p(dev_status), _stream(stream)))


def varlen_desc(t: torch.Tensor) -> Varlen:
    """Descriptor of a contiguous bf16 flat cache [L][2][T_cap][H][D]."""
    if t.dim() != 5 or t.shape[1] != 2:
        raise ValueError("flat cache must be [L][2][T_cap][H][D]")
    if t.dtype != torch.bfloat16 or not t.is_contiguous() or not t.is_cuda:
        raise ValueError("flat cache must be a contiguous bfloat16 device tensor")
    L, _, T, H, D = t.shape
    return Varlen(t.data_ptr(), L, H, D, T)


def specdec_varlen_rollback(src, dst, cu_in, n_acc, k: int, max_len: int, cu_out, pos=None, dev_status=None,
                            stream=None) -> None:
    """Family B rollback: compaction of a flat cache by cumulative lengths."""
    s, d = varlen_desc(src), varlen_desc(dst)
    B = cu_in.numel() - 1
    _req("cu_in", cu_in, (B + 1,), torch.int32)
    _req("n_acc", n_acc, (B,), torch.int32)
    _req("cu_out", cu_out, (B + 1,), torch.int32)
    _req("pos", pos, (pos.numel() if pos is not None else 0,), torch.int64, optional=True)
    _req("dev_status", dev_status, (1,), torch.int32, optional=True)
    _check(lib.specdec_varlen_rollback(ctypes.byref(s), ctypes.byref(d), _p(cu_in), _p(n_acc), B, k, max_len,
                                       _p(cu_out), _p(pos), pos.numel() if pos is not None else 0, _p(dev_status),
                                       _stream(stream)))


def timing_enable(on=True) -> None:
    """True / False for all kernels, or a mask of (1 << KERNEL_*) bits."""
    mask = TIMING_ALL if on is True else (0 if on is False else int(on))
    _check(lib.specdec_timing_enable(mask))


def timing_reset() -> None:
    _check(lib.specdec_timing_reset())


def timing_query(kernel: int) -> tuple[float, int]:
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib.specdec_timing_query(kernel, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


class StepBuffers:
    """Device outputs of one step for B rows, k drafts, a vocabulary of V and a
    pos/mask stride."""

    def __init__(self, B: int, k: int, V: int, pm_cap: int, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        self.tokens = torch.empty((B, k + 1), **i32)
        self.n_acc = torch.empty(B, **i32)
        self.bonus = torch.empty(B, **i32)
        self.pad_out = torch.empty(B, **i32)
        self.w_new = torch.empty(1, **i32)
        self.pos = torch.empty((B, pm_cap), dtype=torch.int64, device=device)
        self.mask = torch.empty((B, pm_cap), dtype=torch.uint8, device=device)
        self.dev_status = torch.zeros(1, **i32)
        self.workspace = alloc_workspace(B, k, V, device)
