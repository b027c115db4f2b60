"""The library's native SequencePool scheduler (specdec_sched_*, host code)
against the oracle's (oracle.exspec.SequencePool): the same batch, lengths,
width and flags at every step of scheduling traces driven by random and
uniform acceptance, eos detection, and the host-side error paths.  No GPU
call is made."""
import numpy as np
import pytest

from oracle.exspec import SequencePool


@pytest.fixture(scope="module")
def sd():
    from paper_2510_22876_amd import specdec
    return specdec


def _run_pair(sd, rng, N, W, B, k, max_new, sort, eos, lens0, p_uniform=0.5, V=9):
    nat = sd.Scheduler(lens0, window=W, batch=B, max_new=max_new, sort_by_length=sort, eos_id=eos)
    orc = SequencePool(list(lens0), window=W, batch=B, max_new=max_new, sort_by_length=sort, eos_id=eos)
    steps = 0
    flags = set()
    for _ in range(4 * N * (max_new + 1) + 2):
        x = nat.next_batch()
        again = nat.next_batch()              # asking twice before a commit returns the same batch
        y = orc.next_batch()
        if y is None:
            assert x is None and again is None and not nat.has_active()
            break
        assert x is not None, "native scheduler stopped early"
        got = (x.slots, x.lens, x.width, x.same_length, x.reuse)
        assert got == (list(y.slots), list(y.lens), y.width, y.same_length, y.reuse), f"step {steps}"
        assert (again.slots, again.reuse) == (x.slots, x.reuse)
        flags.add((x.same_length, x.reuse))
        if rng.random() < p_uniform:
            n_acc = np.full(len(x.slots), int(rng.integers(0, k + 1)), np.int32)
        else:
            n_acc = rng.integers(0, k + 1, size=len(x.slots)).astype(np.int32)
        appended = [list(rng.integers(0, V, size=int(a) + 1)) for a in n_acc]
        nat.commit(x, n_acc, appended)
        orc.commit(y, n_acc, appended)
        assert nat.lengths() == orc.lengths()
        assert nat.has_active() == orc.has_active()
        steps += 1
    else:
        raise AssertionError("the schedule did not finish")
    return steps, flags


@pytest.mark.parametrize("seed", range(40))
def test_native_scheduler_matches_oracle(sd, seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 40))
    W = int(rng.integers(1, 16))
    B = int(rng.integers(1, W + 2))            # batch may exceed the window
    k = int(rng.integers(0, 6))
    max_new = int(rng.integers(1, 24))
    sort = bool(seed % 3)
    eos = int(rng.integers(0, 9)) if seed % 4 == 0 else -1
    spread = [3, 8, 40][seed % 3]
    lens0 = rng.integers(0, spread, size=N)
    _run_pair(sd, rng, N, W, B, k, max_new, sort, eos, lens0)


def test_scheduler_visits_every_decision(sd):
    """Traces that contain reuse, same-length grouping and the padded
    fallback, all matching the oracle."""
    rng = np.random.default_rng(7)
    seen = set()
    for trial in range(12):
        lens0 = rng.integers(10, 14, size=30)
        _, flags = _run_pair(sd, rng, 30, 10, 4, 3, 15, True, -1, lens0, p_uniform=0.7)
        seen |= flags
    assert (True, True) in seen and (True, False) in seen and (False, False) in seen


def test_scheduler_large_pool(sd):
    rng = np.random.default_rng(11)
    lens0 = rng.integers(64, 4096, size=2000)
    steps, _ = _run_pair(sd, rng, 2000, 64, 32, 7, 8, True, -1, lens0, p_uniform=0.3)
    assert steps > 0


def test_scheduler_empty_pool(sd):
    s = sd.Scheduler([], window=4, batch=2, max_new=3)
    assert s.next_batch() is None and not s.has_active() and s.lengths() == []


def test_scheduler_rejects(sd):
    import ctypes
    h = ctypes.c_void_p(None)
    lens = np.array([3, 4], np.int32)
    P = lens.ctypes.data
    lib = sd.lib
    assert lib.specdec_sched_create(P, 2, 0, 1, 1, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    assert lib.specdec_sched_create(P, 2, 1, 0, 1, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    assert lib.specdec_sched_create(P, 2, 1, 1, 0, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    assert lib.specdec_sched_create(None, 2, 1, 1, 1, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    assert lib.specdec_sched_create(P, -1, 1, 1, 1, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    bad = np.array([3, -1], np.int32)
    assert lib.specdec_sched_create(bad.ctypes.data, 2, 1, 1, 1, 1, -1, ctypes.byref(h)) == sd.ERR_INVALID_ARGUMENT
    assert lib.specdec_sched_create(P, 2, 1, 1, 1, 1, -1, None) == sd.ERR_INVALID_ARGUMENT
    assert not h.value
    s = sd.Scheduler(lens, window=2, batch=2, max_new=5, eos_id=3)
    na = np.array([1, 1], np.int32)
    # commit before a batch was handed out
    assert lib.specdec_sched_commit(s._h, na.ctypes.data, None, 2) == sd.ERR_INVALID_ARGUMENT
    b = s.next_batch()
    assert b is not None and b.slots == [0, 1]
    # eos detection needs the tokens; n_acc must lie in [0, k]
    assert lib.specdec_sched_commit(s._h, na.ctypes.data, None, 2) == sd.ERR_INVALID_ARGUMENT
    tok = np.zeros((2, 3), np.int32)
    assert lib.specdec_sched_commit(s._h, na.ctypes.data, tok.ctypes.data, 0) == sd.ERR_INVALID_ARGUMENT
    assert "n_acc" in lib.specdec_last_error().decode()
    assert s.lengths() == [3, 4], "a rejected commit changes nothing"
    tok[1, 1] = 3                                          # row 1 appends eos
    assert lib.specdec_sched_commit(s._h, na.ctypes.data, tok.ctypes.data, 2) == sd.OK
    assert s.lengths() == [5, 6]
    b2 = s.next_batch()
    assert b2.slots == [0] and not b2.reuse               # row 1 finished at eos


def test_native_scheduler_golden_bucket_choice(sd):
    """The native scheduler takes the hand-derived batches of
    tests/golden/sched_bucket_choice.txt (same-length grouping of Alg. 2's
    GetBatch: oldest member's bucket, else the largest, ties to the shorter
    length, else the first window members)."""
    from tests import pins
    g = pins._read_golden("sched_bucket_choice.txt")
    for c in sorted({key.split("_", 1)[0] for key in g}):
        lens0 = g[f"{c}_lens"]
        s = sd.Scheduler(lens0, window=g[f"{c}_window"][0], batch=g[f"{c}_batch"][0], max_new=1, sort_by_length=False)
        b = s.next_batch()
        assert b is not None and b.slots == g[f"{c}_slots"], (c, b.slots if b else None)
        assert b.lens == [lens0[x] for x in b.slots] and not b.reuse
