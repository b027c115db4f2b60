"""A deterministic stand-in for the target and draft models of a speculative
decoding loop, for end-to-end tests of output equivalence (Corollary B.2:
with I1 and I2 maintained, batched speculative greedy decoding produces what
sequential greedy decoding produces).

It plays the model forward pass only and holds none of the method's own
arithmetic (no argmax, no prefix match, no width rule, no cache movement).

* Every token prefix has a 64-bit rolling hash: h(t_0..t_j) = mix(h(t_0..t_{j-1})
  + t_j + 1), from a fixed start value.
* The target model's greedy next token after a prefix is f(h) in [1, V); token
  0 is never produced by a correct forward, so the model emits it as a
  "poison" token when it finds its inputs inconsistent.
* The draft model proposes f(h) with probability ``accept``, else another
  token (the draft model does not look at the cache).
* The cache entry of the token at position j is a bf16 bit pattern derived from
  (h(t_0..t_j), layer, K/V, head, channel), finite and nonzero.
* A verify-window forward checks the batch it is given: the cached columns of
  each row must hold the entries of that row's own tokens, the padding
  columns must be masked, and the position ids of the window must continue the
  row's content.  On any mismatch the row's logits put their maximum on the
  poison token, so a broken cache, mask or position id shows up as a changed
  output, as in a real model.
"""
from __future__ import annotations

import numpy as np

_M64 = (1 << 64) - 1
_START = 0x9E3779B97F4A7C15
POISON = 0


def mix(x):
    """splitmix64's finaliser (Steele, Lea and Flood, 2014), on numpy uint64
    arrays or Python ints."""
    if isinstance(x, int):
        x &= _M64
        x = ((x ^ (x >> 30)) * 0xBF58476D1CE4E5B9) & _M64
        x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & _M64
        return x ^ (x >> 31)
    x = np.asarray(x, np.uint64)
    with np.errstate(over="ignore"):
        x = (x ^ (x >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        x = (x ^ (x >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return x ^ (x >> np.uint64(31))


def prefix_hashes(tokens) -> list:
    """h after each token of the list."""
    out, h = [], _START
    for t in tokens:
        h = mix((h + int(t) + 1) & _M64)
        out.append(h)
    return out


class ToyModel:
    def __init__(self, V: int, n_layers: int, H: int, D: int, accept: float = 0.7, salt: int = 0):
        if V < 3:
            raise ValueError("V >= 3")
        self.V, self.L, self.H, self.D = V, n_layers, H, D
        self.accept = accept
        self.salt = salt
        # (layer, K/V, head, channel) codes of one column, laid out [L][2][H][D]
        l, kv, h, d = np.meshgrid(np.arange(n_layers), np.arange(2), np.arange(H), np.arange(D), indexing="ij")
        self._lane = (((l.astype(np.uint64) * np.uint64(2) + kv.astype(np.uint64)) * np.uint64(H)
                       + h.astype(np.uint64)) * np.uint64(D) + d.astype(np.uint64) + np.uint64(1))
        self._entries: dict = {}

    # ---- the target and draft "models" ----------------------------------------------

    def target_next(self, h: int) -> int:
        return 1 + int(mix(h ^ self.salt) % (self.V - 1))

    def draft_next(self, h: int) -> int:
        u = mix(h ^ 0xD1B54A32D192ED03 ^ self.salt)
        if (u >> 11) / float(1 << 53) < self.accept:
            return self.target_next(h)
        alt = 1 + int(mix(u) % (self.V - 1))
        return alt if alt != self.target_next(h) else 1 + (alt % (self.V - 1))

    def entry(self, h: int) -> np.ndarray:
        """Cache entry [L][2][H][D] (uint16 bf16 bits) of the token whose prefix
        hash is h: finite (exponent below 0xFF) and nonzero."""
        e = self._entries.get(h)
        if e is None:
            with np.errstate(over="ignore"):
                m = mix(self._lane * np.uint64(0x2545F4914F6CDD1D) ^ np.uint64(h))
            e = ((m & np.uint64(0xBFFF)) | np.uint64(1)).astype(np.uint16)
            e.setflags(write=False)
            self._entries[h] = e
        return e

    # ---- sequential greedy decoding (the reference of Corollary B.2) -----------------

    def greedy(self, prompt, n_new: int) -> list:
        seq = list(prompt)
        h = prefix_hashes(seq)[-1]
        for _ in range(n_new):
            t = self.target_next(h)
            seq.append(t)
            h = mix((h + t + 1) & _M64)
        return seq[len(prompt):]

    # ---- one speculative round on a left-padded batch ---------------------------------

    def draft(self, row_tokens, k: int) -> list:
        """k draft tokens after the row's content tokens (cached + pending)."""
        h = prefix_hashes(row_tokens)[-1]
        out = []
        for _ in range(k):
            t = self.draft_next(h)
            out.append(t)
            h = mix((h + t + 1) & _M64)
        return out

    def forward_window(self, kv_row, pad: int, width: int, row_tokens, drafts, pos_row, mask_row,
                       V_out: int | None = None):
        """The verify forward of one row: kv_row [L][2][H][cap][D] uint16 holds
        the batch cache (content at [pad, width)), row_tokens its content
        tokens (cached + pending), drafts its k drafts, pos_row/mask_row the
        position ids and mask over [0, width + k + 1).  Returns the window's
        cache entries [L][2][H][k+1][D] and the logits [k+1][V] (fp32; maximum
        1.0 on the predicted token, poison on inconsistency)."""
        k = len(drafts)
        n = len(row_tokens) - 1                      # cached tokens
        ok = width - pad == n
        hs = prefix_hashes(list(row_tokens) + list(drafts))
        if ok:
            for j in range(n):                       # the cached columns
                if not np.array_equal(kv_row[:, :, :, pad + j, :], self.entry(hs[j])):
                    ok = False
                    break
        if ok:
            m = np.asarray(mask_row[: width + k + 1])
            ok = bool(np.all(m[:pad] == 0) and np.all(m[pad:] == 1))
        if ok:
            p = np.asarray(pos_row[width: width + k + 1])
            ok = bool(np.array_equal(p, np.arange(n, n + k + 1)))
        window = np.stack([self.entry(hs[n + r]) for r in range(k + 1)], axis=3)
        V = V_out or self.V
        logits = np.zeros((k + 1, V), np.float32)
        for r in range(k + 1):
            logits[r, self.target_next(hs[n + r]) if ok else POISON] = 1.0
        return window, logits
