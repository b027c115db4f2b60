"""ctypes binding of libspecdec.so (C ABI in include/specdec.h).

Argument marshalling only: torch tensors are passed as device pointers, the
stream is torch's current HIP stream, and every step of the path runs in the
library's HIP kernels.  Importing this module loads the library and raises if
it has not been built; there is no fallback.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

_LIB_PATH = Path(__file__).resolve().parent / "libspecdec.so"

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_HIP, ERR_WORKSPACE = 0, 1, 2, 3, 4
F32, BF16, F16 = 0, 1, 2
DTYPE_OF = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}
KERNEL_VERIFY, KERNEL_REALIGN, KERNEL_POSMASK = 0, 1, 2
TIMING_ALL = 7
DEV_BAD_PAD_IN, DEV_BAD_ACCEPT, DEV_BAD_WIDTH, DEV_BAD_PAD_OUT = 1, 2, 4, 8

EXPORTED = (
    "specdec_abi_version", "specdec_last_error", "specdec_workspace_bytes", "specdec_workspace_init",
    "specdec_verify_greedy", "specdec_realign_kv", "specdec_build_posmask", "specdec_realign_tokens",
    "specdec_step",
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
    lib.specdec_timing_enable.argtypes = [i32]
    lib.specdec_timing_query.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    for name in ("specdec_workspace_init", "specdec_verify_greedy", "specdec_realign_kv",
                 "specdec_build_posmask", "specdec_realign_tokens", "specdec_step", "specdec_timing_enable",
                 "specdec_timing_reset", "specdec_timing_query"):
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


def specdec_step(logits, draft, pad_in, W_in: int, src, dst, tokens, n_acc, bonus, pad_out, w_new,
                 pos, mask, workspace, dev_status=None, sync_w_new: bool = False, stream=None,
                 s_in=None, s_out=None, pad_id: int = 0):
    """The fused step (with the token row S when ``s_in`` / ``s_out`` are
    given); returns L' as a Python int when ``sync_w_new``."""
    B, kp1, V = logits.shape
    _check_verify(logits, draft, pad_in, tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status)
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
    _check(lib.specdec_step(
        _p(logits), DTYPE_OF[logits.dtype], _p(draft), _p(pad_in), B, kp1 - 1, V, W_in,
        ctypes.byref(s), ctypes.byref(d), _p(tokens), _p(n_acc), _p(bonus), _p(pad_out), _p(w_new),
        _p(pos), _p(mask), pos.shape[1], _p(s_in), s_in.shape[1] if s_in is not None else 0, _p(s_out),
        s_out.shape[1] if s_out is not None else 0, pad_id,
        _p(workspace), workspace.numel() * workspace.element_size(),
        _p(dev_status), ctypes.byref(host) if sync_w_new else None, _stream(stream)))
    return host.value if sync_w_new else None


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
