"""End-to-end decoding loops over a toy model (``toy_model.ToyModel``), used
to check Corollary B.2 (output equivalence with sequential greedy decoding)
for both batching algorithms of arXiv 2510.22876:

* ``run_exspec``: Algorithm 2 (EXSpec): a pool of unpadded sequences, a
  scheduler that forms batches over a sliding window, batch gather, verify,
  write-back.
* ``run_eqspec``: Algorithm 1 (EqSpec): fixed batches realigned after every
  verification (unpad-append-repad of cache and token row, I2 positions).

The loops only sequence the steps; every step is delegated to a backend: the
oracle (``OracleBackend``, numpy on the CPU) or the HIP library
(``tests/gpu_util.HipBackend``).  The scheduler is passed in: the oracle's
``oracle.exspec.SequencePool`` or the library's native one.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import oracle
from tests.toy_model import ToyModel, prefix_hashes

PAD_ID = -2
TOK_FILL = -7


@dataclass
class LoopResult:
    generated: list                      # per sequence: its generated tokens
    trace: list = field(default_factory=list)   # per step: (slots, width, reuse, same_length, n_acc)
    pool: np.ndarray | None = None       # final pool cache (uint16 bits)
    pool_tok: np.ndarray | None = None
    lens: np.ndarray | None = None


class OracleBackend:
    """Every step of the method on the CPU oracle (numpy arrays)."""

    def to_host(self, x):
        return x

    def from_host(self, x):
        return x

    def gather(self, pool, pool_tok, lens, slots, Lb, batch_cap, btok_stride, pad_id):
        return oracle.gather_batch(pool, pool_tok, lens, slots, Lb, batch_cap, btok_stride, pad_id)

    def posmask(self, pads, width, k, pm_cap):
        return oracle.posmask(pads, width, k, pm_cap)

    def write_window(self, batch, row, col, entries):
        batch[:, :, row, :, col: col + entries.shape[3], :] = entries

    def verify(self, logits, draft, pads, W_in):
        return oracle.verify(logits, "f32", draft, pads, W_in)

    def rollback(self, tokens, n_acc, pads, W_in):
        return oracle.rollback(tokens, n_acc, pads, W_in)

    def scatter(self, batch, pads, tokens, n_acc, slots, Lb, pool, pool_tok, lens, batch_tok):
        oracle.scatter_accepted(batch, pads, tokens, n_acc, slots, Lb, pool, pool_tok, lens, batch_tok)

    def realign(self, kv, k, W_in, pads, n_acc, w_new, tokens, s, pad_id):
        out = oracle.realign_kv(kv, k, W_in, pads, n_acc, w_new, dst=np.zeros_like(kv))
        s_out = oracle.realign_tokens(s, tokens, pads, n_acc, w_new, W_in, pad_id, out_stride=s.shape[1])
        return out, s_out


def init_pool(model: ToyModel, prompts, cap: int, tok_stride: int):
    """Prefill: slot s caches the entries of all but the last prompt token;
    the last one is the pending token."""
    N = len(prompts)
    pool = np.zeros((model.L, 2, N, model.H, cap, model.D), np.uint16)
    pool_tok = np.full((N, tok_stride), TOK_FILL, np.int32)
    lens = np.zeros(N, np.int32)
    for s, p in enumerate(prompts):
        pool_tok[s, : len(p)] = p
        hs = prefix_hashes(p)
        for j in range(len(p) - 1):
            pool[:, :, s, :, j, :] = model.entry(hs[j])
        lens[s] = len(p) - 1
    return pool, pool_tok, lens


def _model_round(model, be, batch, btok, pads, Lb, k, pos, mask):
    """Draft and target forward of one round over a batch (on host copies)."""
    kv_h = be.to_host(batch)
    tok_h = be.to_host(btok)
    pos_h, mask_h = be.to_host(pos), be.to_host(mask)
    B = len(pads)
    draft = np.zeros((B, k), np.int32)
    logits = np.zeros((B, k + 1, model.V), np.float32)
    for i in range(B):
        row_tokens = [int(t) for t in tok_h[i, int(pads[i]): Lb + 1]]
        d = model.draft(row_tokens, k)
        win, lg = model.forward_window(kv_h[:, :, i], int(pads[i]), Lb, row_tokens, d, pos_h[i], mask_h[i])
        be.write_window(batch, i, Lb, win)
        draft[i] = d
        logits[i] = lg
    return draft, logits


def run_exspec(be, model: ToyModel, prompts, sched, k: int, max_new: int) -> LoopResult:
    """Algorithm 2 with the scheduler ``sched`` (next_batch / commit)."""
    N = len(prompts)
    maxp = max(len(p) for p in prompts)
    cap = maxp + max_new + k + 1
    bcap = cap + k + 1
    pool, pool_tok, lens = init_pool(model, prompts, cap, cap + 2)
    pool_d, pool_tok_d, lens_d = be.from_host(pool), be.from_host(pool_tok), be.from_host(lens)
    batch = btok = pads = None
    trace = []
    for _ in range(10 * N * max_new + 10):
        b = sched.next_batch()
        if b is None:
            break
        slots = np.asarray(b.slots, np.int32)
        Lb = int(b.width)
        if not b.reuse:
            batch, btok, pads = be.gather(pool_d, pool_tok_d, lens_d, be.from_host(slots), Lb, bcap, bcap + 1, PAD_ID)
        pads_h = np.asarray(be.to_host(pads), np.int32)
        pos, mask = be.posmask(pads, Lb, k, bcap + 1)
        draft, logits = _model_round(model, be, batch, btok, pads_h, Lb, k, pos, mask)
        v = be.verify(be.from_host(logits), be.from_host(draft), pads, Lb + k + 1)
        be.scatter(batch, pads, v["tokens"], v["n_acc"], be.from_host(slots), Lb, pool_d, pool_tok_d, lens_d, btok)
        n_acc = np.asarray(be.to_host(v["n_acc"]), np.int32)
        toks = np.asarray(be.to_host(v["tokens"]), np.int32)
        sched.commit(b, n_acc, [toks[i, : n_acc[i] + 1] for i in range(len(slots))])
        assert list(sched.lengths()) == [int(x) for x in np.asarray(be.to_host(lens_d))], "pool lengths diverged"
        trace.append((list(b.slots), Lb, bool(b.reuse), bool(b.same_length), [int(x) for x in n_acc]))
    else:
        raise AssertionError("the scheduler did not finish")
    pool_h, tok_h, lens_h = be.to_host(pool_d), be.to_host(pool_tok_d), np.asarray(be.to_host(lens_d))
    gen = [list(tok_h[s, len(p): int(lens_h[s]) + 1]) for s, p in enumerate(prompts)]
    return LoopResult(gen, trace, pool_h, tok_h, lens_h)


def run_eqspec(be, model: ToyModel, prompts, B: int, k: int, max_new: int, rollback: bool = False) -> LoopResult:
    """Algorithm 1: consecutive groups of B prompts, each decoded as one fixed
    batch, realigned after every verification, until every row has generated
    max_new tokens.  With ``rollback`` every round is truncated to the batch's
    minimum accepted count first (Family A rollback); the trace then records
    the accepted counts before truncation."""
    gen = [None] * len(prompts)
    trace = []
    for g0 in range(0, len(prompts), B):
        group = prompts[g0: g0 + B]
        nb = len(group)
        n = np.array([len(p) - 1 for p in group], np.int32)
        W0 = int(n.max())
        cap = W0 + (k + 1) * (max_new + 1) + k + 1   # the widest row can gain k+1 a step
        pads = (W0 - n).astype(np.int32)
        kv = np.zeros((model.L, 2, nb, model.H, cap, model.D), np.uint16)
        s = np.full((nb, cap + 2), PAD_ID, np.int32)
        for i, p in enumerate(group):
            hs = prefix_hashes(p)
            for j in range(len(p) - 1):
                kv[:, :, i, :, pads[i] + j, :] = model.entry(hs[j])
            s[i, pads[i]: W0 + 1] = p
        kv_d, s_d, pads_d = be.from_host(kv), be.from_host(s), be.from_host(pads)
        made = np.zeros(nb, np.int64)
        while made.min() < max_new:
            pos, mask = be.posmask(pads_d, W0, k, cap + 1)
            draft, logits = _model_round(model, be, kv_d, s_d, np.asarray(be.to_host(pads_d)), W0, k, pos, mask)
            W_in = W0 + k + 1
            v = be.verify(be.from_host(logits), be.from_host(draft), pads_d, W_in)
            if rollback:
                verified = np.asarray(be.to_host(v["n_acc"]), np.int32)
                v = dict(v, **be.rollback(v["tokens"], v["n_acc"], pads_d, W_in))
            w_new = int(np.asarray(be.to_host(v["w_new"])).reshape(-1)[0])
            kv_d, s_d = be.realign(kv_d, k, W_in, pads_d, v["n_acc"], v["w_new"], v["tokens"], s_d, PAD_ID)
            n_acc = np.asarray(be.to_host(v["n_acc"]), np.int32)
            made += n_acc + 1
            trace.append((list(range(g0, g0 + nb)), W0, False, False,
                          [int(x) for x in (verified if rollback else n_acc)]))
            pads_d = v["pad_out"]
            W0 = w_new
            if W0 + k + 1 > cap:
                raise AssertionError("cache capacity exceeded")
        s_h = be.to_host(s_d)
        pads_h = np.asarray(be.to_host(pads_d))
        for i, p in enumerate(group):
            gen[g0 + i] = list(s_h[i, int(pads_h[i]) + len(p): W0 + 1])
    return LoopResult(gen, trace)


def check_equivalence(model: ToyModel, prompts, res: LoopResult, max_new: int):
    """Corollary B.2: each sequence's generated tokens are what sequential
    greedy decoding produces (as many as the loop generated, at least
    max_new)."""
    for s, p in enumerate(prompts):
        got = [int(t) for t in res.generated[s]]
        assert len(got) >= max_new, (s, len(got))
        want = model.greedy(p, len(got))
        assert got == want, f"sequence {s}: first difference at {next(i for i in range(len(got)) if got[i] != want[i])}"


def check_pool_cache(model: ToyModel, prompts, res: LoopResult):
    """After the loop every slot caches exactly the entries of its own tokens
    (all but the pending last one)."""
    for s in range(len(prompts)):
        n = int(res.lens[s])
        toks = [int(t) for t in res.pool_tok[s, : n + 1]]
        hs = prefix_hashes(toks)
        for j in range(n):
            assert np.array_equal(res.pool[:, :, s, :, j, :], model.entry(hs[j])), (s, j)


def random_prompts(rng, N: int, lo: int, hi: int, V: int, equal_groups: int = 0):
    """N prompts of lengths U[lo, hi]; with equal_groups > 0 the lengths come
    from that many distinct values (so same-length groups exist)."""
    if equal_groups:
        choices = rng.integers(lo, hi + 1, size=equal_groups)
        lens = rng.choice(choices, size=N)
    else:
        lens = rng.integers(lo, hi + 1, size=N)
    return [[int(t) for t in rng.integers(1, V, size=int(n))] for n in lens]
