"""GPU parity on seeded random configurations.

Each case draws its shape and recipe from a fixed seed, so the set is the
same on every run: batch size, draft count, vocabulary (1 to 128256, aligned
and ragged), logit dtype, cache layers / heads / head size, prompt length
distribution, acceptance pattern, planted ties, left-padding slack (the
smallest padding above 0: shifts of both signs), spare capacity, the
out-of-place or in-place variant, the fused or split entry points and the
token row.  The greedy step is compared with the oracle element by element
(tokens, counts, width, paddings, every cache byte, positions, mask, token
row); stochastic verification, the EXSpec gather and the Family B compaction
go through the same checks as their hand-picked cases.
"""
import numpy as np
import pytest
import torch

from paper_2510_22876_amd import workloads as wl
from tests.gpu_util import run_gpu, say
from tests.test_gpu_exspec import test_gather_matches_oracle as _gather_case
from tests.test_gpu_parity import _full_check
from tests.test_gpu_rollback import test_varlen_rollback_matches_oracle as _varlen_case
from tests.test_gpu_sample import test_verify_sample_matches_oracle as _sample_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2510_22876_amd import specdec
    yield specdec
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _greedy_case(seed):
    r = np.random.default_rng([seed, 77])
    B = int(r.choice([1, 2, 3, 5, 8, 13, 31, 64]))
    k = int(r.integers(0, 9))
    V = int(r.choice([1, 2, 7, 100, 1001, 4096, 32000, 50257, 128256]))
    dt = str(r.choice(["f32", "bf16", "f16"]))
    L, H, D = int(r.integers(1, 4)), int(r.integers(1, 5)), int(8 * r.integers(1, 33))
    lo = int(r.integers(1, 64))
    hi = lo + int(r.integers(0, 700))
    prompt = [("uniform", lo, hi), ("loguniform", lo, hi), ("fixed", lo)][int(r.integers(0, 3))]
    accept = [("uniform",), ("trunc_geom", 0.6), ("alternate",), ("fixed", int(r.integers(0, k + 1)))][
        int(r.integers(0, 4))]
    w = wl.Workload(f"rand{seed}", B, k, V, dt, 2.0, L, H, D, prompt, accept,
                    tie_frac=float(r.choice([0.0, 0.0, 0.3])), extra_cap=int(r.integers(0, 6)))
    if r.random() < 0.3:                   # the smallest padding above 0
        n = wl.prompt_lengths(w, seed)
        w = w.scaled(W_in=int(n.max()) + k + 1 + int(r.integers(1, 40)))
    variant = str(r.choice(["oop", "inplace"]))
    api = str(r.choice(["step", "split"]))
    tokens = [None, "oop", "inplace"][int(r.integers(0, 3))]
    return w, variant, api, tokens


@pytest.mark.parametrize("seed", range(200))
def test_random_greedy_step(sd, seed):
    w, variant, api, tokens = _greedy_case(seed)
    say(f"random step {seed}: {w} variant={variant} api={api} tokens={tokens}")
    _full_check(run_gpu(w, seed=seed, variant=variant, api=api, tokens=tokens))


def _sample_params(seed):
    r = np.random.default_rng([seed, 78])
    return (int(r.choice([1, 3, 8, 17])), int(r.integers(0, 9)), int(r.choice([1, 5, 100, 1000, 32000, 65539])),
            str(r.choice(["f32", "bf16", "f16"])), float(r.choice([0.3, 0.7, 1.0, 1.7])),
            str(r.choice(["sampled", "sampled", "uniform", "greedy"])))


@pytest.mark.parametrize("seed", range(60))
def test_random_verify_sample(sd, seed):
    _sample_case(sd, _sample_params(seed), seed)


def _gather_params(seed):
    r = np.random.default_rng([seed, 79])
    N = int(r.integers(1, 13))
    return (int(r.integers(1, 3)), int(r.integers(1, 4)), int(8 * r.integers(1, 33)), N, int(r.integers(1, N + 1)),
            int(r.integers(0, 301)), bool(r.random() < 0.3), int(r.integers(0, 6)), int(r.integers(0, 9)))


@pytest.mark.parametrize("seed", range(60))
def test_random_gather(sd, seed):
    _gather_case(sd, _gather_params(seed), seed % 2)


def _varlen_params(seed):
    r = np.random.default_rng([seed, 80])
    return (int(r.integers(1, 65)), int(r.integers(0, 9)), int(r.integers(1, 3)), int(r.integers(1, 5)),
            int(8 * r.integers(1, 17)))


@pytest.mark.parametrize("seed", range(60))
def test_random_varlen_rollback(sd, seed):
    _varlen_case(sd, _varlen_params(seed), int(np.random.default_rng([seed, 81]).choice([0, 30])))
