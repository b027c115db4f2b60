"""Oracle of EXSpec's cross-batch scheduling (arXiv 2510.22876, Algorithm 2,
Appendix "EXSpec: Cross-Batch Scheduling Algorithm"; Section 3.2,
"Cross-Batch Scheduling").

TEST INFRASTRUCTURE ONLY: a plain Python statement of the scheduling
decisions the library's native scheduler must reproduce exactly.

The paper fixes the structure (a pool of ragged sequences, a sliding window of
W > B active sequences, same-length batches concatenated without padding,
lazy realignment, unpad-repad as the fallback, write-back of accepted tokens
and cache entries, deactivation of finished sequences, window refill) but not
the policy inside it.  Readings taken here:

* Pool order: sequences sorted by prompt length (ties by index) when
  ``sort_by_length``, else in input order.  The window is the first W active
  sequences in pool order.
* Lazy realignment: the previous batch is reused unchanged when its last step
  accepted the same number of drafts in every row (so every offset of Eq. (2)
  is zero, Corollary B.4, and the batch is still rectangular) and all its rows
  are still active and in the window.
* Same-length grouping: window members are bucketed by their current length
  (cached entries).  The bucket holding the oldest window member (first in
  pool order) is used when it has at least B members, else the largest bucket
  with at least B members (ties: the shorter length); its first B members in
  pool order form the batch.
* Fallback (unpad-repad): the first B window members in pool order.
* Batch width: the longest row's length (equal lengths: no padding).
* Completion: a sequence is deactivated once it has generated at least
  ``max_new`` tokens, or appended ``eos_id`` (when eos_id >= 0).
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass
class Batch:
    slots: list        # pool slots of the rows, in row order
    lens: list         # their lengths (cached entries) when the batch was formed
    width: int         # Lb: the longest row's length
    same_length: bool  # every row has the same length (no padding)
    reuse: bool        # the previous batch, unchanged (no gather needed)


class SequencePool:
    def __init__(self, prompt_lens, window: int, batch: int, max_new: int, sort_by_length: bool = True,
                 eos_id: int = -1):
        n = len(prompt_lens)
        if window < 1 or batch < 1:
            raise ValueError("window and batch must be positive")
        self.N = n
        self.W = window
        self.B = batch
        self.max_new = max_new
        self.eos_id = eos_id
        self.order = sorted(range(n), key=lambda s: (prompt_lens[s], s)) if sort_by_length else list(range(n))
        self.len = [int(x) for x in prompt_lens]
        self.generated = [0] * n
        self.active = [True] * n
        self.prev: list | None = None      # previous batch if still rectangular

    def has_active(self) -> bool:
        return any(self.active)

    def lengths(self) -> list:
        return list(self.len)

    def window(self) -> list:
        return [s for s in self.order if self.active[s]][: self.W]

    def next_batch(self) -> Batch | None:
        win = self.window()
        if not win:
            return None
        # (members of the previous batch that are all still active are still
        # in the window: deactivations only move later sequences forward)
        if self.prev is not None and all(self.active[s] for s in self.prev):
            lens = [self.len[s] for s in self.prev]
            return Batch(list(self.prev), lens, max(lens), len(set(lens)) == 1, True)
        B = min(self.B, len(win))
        buckets: dict[int, list] = {}
        for s in win:
            buckets.setdefault(self.len[s], []).append(s)
        first = buckets[self.len[win[0]]]
        chosen = None
        if len(first) >= B:
            chosen = first[:B]
        else:
            big = [b for b in buckets.values() if len(b) >= B]
            if big:
                best = max(big, key=lambda b: (len(b), -self.len[b[0]]))
                chosen = best[:B]
        if chosen is not None:
            lens = [self.len[s] for s in chosen]
            return Batch(chosen, lens, lens[0], True, False)
        chosen = win[:B]
        lens = [self.len[s] for s in chosen]
        return Batch(chosen, lens, max(lens), len(set(lens)) == 1, False)

    def commit(self, batch: Batch, n_acc, appended) -> None:
        """Write-back bookkeeping after verification (Alg. 2, Phase 4):
        appended[i] are the n_acc[i]+1 tokens row i gained."""
        for i, s in enumerate(batch.slots):
            a = int(n_acc[i]) + 1
            self.len[s] += a
            self.generated[s] += a
            if self.generated[s] >= self.max_new or (self.eos_id >= 0 and self.eos_id in list(appended[i])):
                self.active[s] = False
        uniform = len({int(x) for x in n_acc}) == 1
        self.prev = list(batch.slots) if uniform else None
